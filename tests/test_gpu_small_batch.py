"""GPU parity of the small-batch GEMV (2 <= m <= 16 activation rows).

bitcos_gemv with m > 1 runs the matrix-core kernel on layouts with one sign
offset per row and whole 128-weight groups, and m batch-1 launches on any
other layout; trit5_gemv and bit2_gemv always take the batch-1 path.  Every
output row of every batch row is compared with the oracle's dense
definition, to the bars of the batch-1 tests (parity_checks.py): raw int32
and per-tensor int8 bit-exact, group or activation scales within
1e-5 sum_g |S a A|, bf16 within 1e-3.
"""

import functools

import numpy as np
import pytest

import oracle as O
import workloads as wl
from parity_checks import (bf16_bound, check_bf16, check_grouped, group_bound, inputs, run, sampled_rows, say,
                           to_dev_x)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
api = pytest.importorskip("paper_2609_16338_amd.api")
from paper_2609_16338_amd import _native as N  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    N.lib()


def _acts(kind, m, k, seed):
    if kind == "int8":
        return wl.act_int8(m, k, wl.rng_for(400, seed, m, k))
    return wl.act_bf16(m, k, wl.rng_for(401, seed, m, k))


def _check(y, w, sc, group, x, kind, xscale=None, raw=False):
    if raw:
        assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32))
        return
    if kind == "bf16":
        ref = O.dense_gemv(w, sc, group, x, x_is_bf16_bits=True)
        check_bf16(y, ref, bf16_bound(w, sc, group, x))
        return
    ref = O.dense_gemv(w, sc, group, x, xscale)
    if group == 0 and xscale is None:
        assert np.array_equal(y, ref)
    else:
        check_grouped(y, ref, group_bound(w, sc, group, x, xscale))


# ---------------------------------------------------------------------------
# Matrix-core kernel: batch sizes, scale modes, ragged shapes
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("m", [2, 3, 4, 7, 16])
def test_small_batch_int8_raw_and_grouped(m):
    n, k = 256, 1024
    w, sc = inputs(n, k, 0.5, 128, 500 + m)
    x = _acts("int8", m, k, 1)
    y, L = run(N.FMT_BITCOS, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW)
    assert L.unit_rows == 1
    _check(y, w, sc, 128, x, "int8", raw=True)
    y, _ = run(N.FMT_BITCOS, w, sc, 128, x, "int8")
    _check(y, w, sc, 128, x, "int8")


@pytest.mark.parametrize("m", [2, 4, 16])
@pytest.mark.parametrize("group", [0, 128])
def test_small_batch_bf16(m, group):
    n, k = 97, 2560
    w, sc = inputs(n, k, 0.42, group, 510 + m)
    x = _acts("bf16", m, k, 2)
    y, _ = run(N.FMT_BITCOS, w, sc, group, x, "bf16")
    _check(y, w, sc, group, x, "bf16")


@pytest.mark.parametrize("m", [2, 16])
def test_small_batch_per_tensor_int8_bit_exact(m):
    n, k = 45, 6912
    w, sc = inputs(n, k, 0.42, 0, 520 + m)
    x = _acts("int8", m, k, 3)
    y, _ = run(N.FMT_BITCOS, w, sc, 0, x, "int8")
    _check(y, w, sc, 0, x, "int8")


@pytest.mark.parametrize("m", [3, 16])
@pytest.mark.parametrize("group", [0, 128])
@pytest.mark.parametrize("k", [2560, 640, 1152])
def test_small_batch_activation_scales(m, group, k):
    # k = 640 and 1152: a group count that is not a multiple of four, so the
    # last step of a unit has groups past the row's end
    n = 70
    w, sc = inputs(n, k, 0.42, group, 530 + m)
    xb = _acts("bf16", m, k, 4)
    q, a = O.quantize_activations(xb)
    y, _ = run(N.FMT_BITCOS, w, sc, group, q, "int8", xscale=a)
    _check(y, w, sc, group, q, "int8", xscale=a)
    y, _ = run(N.FMT_BITCOS, w, sc, group, q, "int8", xscale=a, y_mode=N.Y_I32_RAW)
    _check(y, w, sc, group, q, "int8", raw=True)


@pytest.mark.parametrize("m", [1, 4, 16])
@pytest.mark.parametrize("group", [0, 128])
def test_small_batch_bf16_activation_scales(m, group):
    """bf16 activations with per-group activation scales, y = sum_g S a A:
    the small-batch kernel's bf16 activation-scale variant (at m = 1 through
    a row too long for the batch-1 kernels)."""
    n, k = (37, 20480) if m == 1 else (70, 2560)
    w, sc = inputs(n, k, 0.42, group, 535 + m)
    xb = _acts("bf16", m, k, 5)
    a = wl.rng_for(536, m, k).uniform(0.5, 2.0, size=(m, k // 128)).astype(np.float32)
    y, L = run(N.FMT_BITCOS, w, sc, group, xb, "bf16", xscale=a)
    assert api.describe(L, m, N.X_BF16).kernel == N.KERNEL_SMALL_BATCH
    ref = O.dense_gemv(w, sc, group, xb, a, x_is_bf16_bits=True)
    check_bf16(y, ref, bf16_bound(w, sc, group, xb) * float(a.max()))


@pytest.mark.parametrize("n,k", [(1, 128), (31, 128), (33, 640), (17, 384), (64, 12288), (5, 25600)])
@pytest.mark.parametrize("kind", ["int8", "bf16"])
def test_small_batch_ragged_shapes(n, k, kind):
    # rows not a multiple of the 32-row unit; groups not a multiple of four
    m = 5
    w, sc = inputs(n, k, 0.45, 128, 540 + n + k)
    x = _acts(kind, m, k, 5)
    if kind == "int8":
        y, _ = run(N.FMT_BITCOS, w, sc, 128, x, kind, y_mode=N.Y_I32_RAW)
        _check(y, w, sc, 128, x, kind, raw=True)
    y, _ = run(N.FMT_BITCOS, w, sc, 128, x, kind)
    _check(y, w, sc, 128, x, kind)


@pytest.mark.parametrize("z", [0.0, 1.0])
def test_small_batch_degenerate_densities(z):
    w, sc = inputs(40, 1024, z, 128, 550)
    w[5, :] = -1
    x = _acts("int8", 8, 1024, 6)
    x[3] = 127
    x[4] = -127
    y, _ = run(N.FMT_BITCOS, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW)
    _check(y, w, sc, 128, x, "int8", raw=True)


def test_small_batch_rows_are_independent():
    """Batch row i of an m-row call equals the batch-1 call on row i (int8 raw: exact)."""
    n, k, m = 130, 4096, 6
    w, sc = inputs(n, k, 0.467, 128, 560)
    x = _acts("int8", m, k, 7)
    y, _ = run(N.FMT_BITCOS, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW)
    for i in range(m):
        yi, _ = run(N.FMT_BITCOS, w, sc, 128, x[i:i + 1], "int8", y_mode=N.Y_I32_RAW)
        assert np.array_equal(y[i:i + 1], yi)


def test_small_batch_deterministic_repeat():
    w, sc = inputs(300, 5120, 0.45, 128, 570)
    xb = _acts("bf16", 16, 5120, 8)
    a, _ = run(N.FMT_BITCOS, w, sc, 128, xb, "bf16")
    b, _ = run(N.FMT_BITCOS, w, sc, 128, xb, "bf16")
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


# ---------------------------------------------------------------------------
# Layouts the matrix-core kernel does not take: m batch-1 launches
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("unit", [2, 7])
def test_small_batch_other_unit_rows(unit):
    w, sc = inputs(45, 2560, 0.45, 128, 580)
    x = _acts("int8", 3, 2560, 9)
    y, L = run(N.FMT_BITCOS, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW, unit=unit)
    assert L.unit_rows == unit
    _check(y, w, sc, 128, x, "int8", raw=True)


def test_small_batch_k_not_multiple_of_128():
    w, sc = inputs(9, 96, 0.4, 0, 590)
    x = _acts("int8", 4, 96, 10)
    y, _ = run(N.FMT_BITCOS, w, sc, 0, x, "int8")
    _check(y, w, sc, 0, x, "int8")


@pytest.mark.parametrize("fmt", [N.FMT_TRIT5, N.FMT_BIT2])
def test_small_batch_baselines(fmt):
    w, sc = inputs(37, 2560, 0.42, 128, 600)
    x = _acts("int8", 4, 2560, 11)
    y, _ = run(fmt, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW)
    _check(y, w, sc, 128, x, "int8", raw=True)
    xb = _acts("bf16", 3, 2560, 12)
    y, _ = run(fmt, w, sc, 128, xb, "bf16")
    _check(y, w, sc, 128, xb, "bf16")


def test_batch_size_out_of_range_is_an_error():
    import ctypes
    w, sc = inputs(8, 256, 0.4, 128, 610)
    L, blob = api.plan_and_pack(N.FMT_BITCOS, w, sc, 128)
    bd = torch.from_numpy(blob).cuda()
    x = torch.zeros((17, 256), dtype=torch.int8, device="cuda")
    y = torch.zeros((17, 8), dtype=torch.float32, device="cuda")
    lib = N.lib()
    for m in (0, 17, -1):
        st = lib.bitcos_gemv(ctypes.byref(L), ctypes.c_void_p(bd.data_ptr()), m, ctypes.c_void_p(x.data_ptr()),
                             N.X_I8, None, ctypes.c_void_p(y.data_ptr()), N.Y_F32, None)
        assert st == N.E_ARG, m


# ---------------------------------------------------------------------------
# Batched launch with m > 1 (mixed shapes in one table)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("kind,group,xscale", [("int8", 128, False), ("int8", 128, True), ("int8", 0, False),
                                               ("bf16", 128, False), ("bf16", 0, False)])
def test_small_batch_table(kind, group, xscale):
    m = 4
    specs = [(64, 2560, 0.42), (7, 5120, 0.0), (300, 1024, 0.5), (33, 640, 1.0), (129, 2560, 0.467)]
    layouts, blobs, xs, ys, xss, cases = [], [], [], [], [], []
    for i, (n, k, z) in enumerate(specs):
        w, sc = inputs(n, k, z, group, 620 + i)
        a_np = None
        if kind == "int8":
            x = _acts("int8", m, k, 20 + i)
            if xscale and i % 2 == 0:        # some GEMVs with activation scales, some without
                x, a_np = O.quantize_activations(_acts("bf16", m, k, 30 + i))
        else:
            x = _acts("bf16", m, k, 40 + i)
        L, blob = api.plan_and_pack(N.FMT_BITCOS, w, sc, group)
        layouts.append(L)
        blobs.append(torch.from_numpy(blob).cuda())
        xs.append(to_dev_x(x, kind))
        xss.append(None if a_np is None else torch.from_numpy(np.ascontiguousarray(a_np, np.float32)).cuda())
        ys.append(torch.full((m, n), -7.0, dtype=torch.float32, device="cuda"))
        cases.append((w, sc, x, a_np))
    say("small-batch table", kind, f"group={group}", "xscale" if xscale else "")
    b = api.Batch(layouts, blobs, xs, ys, xss if xscale else None)
    assert b.m == m
    b.run()
    torch.cuda.synchronize()
    first = []
    for y, (w, sc, x, a_np) in zip(ys, cases):
        got = y.cpu().numpy()
        _check(got, w, sc, group, x, kind, xscale=a_np)
        first.append(got.copy())
    b.run()
    torch.cuda.synchronize()
    for y, f in zip(ys, first):
        assert np.array_equal(y.cpu().numpy().view(np.uint32), f.view(np.uint32))


def test_small_batch_table_rejects_other_layouts():
    w, sc = inputs(8, 2560, 0.4, 128, 640)
    L1, b1 = api.plan_and_pack(N.FMT_BITCOS, w, sc, 128)
    L2, b2 = api.plan_and_pack(N.FMT_BITCOS, w, sc, 128, 4)      # 4 rows per sign offset
    L3, b3 = api.plan_and_pack(N.FMT_TRIT5, w, sc, 128)
    dev = lambda a: torch.from_numpy(a).cuda()  # noqa: E731
    x = torch.zeros((2, 2560), dtype=torch.int8, device="cuda")
    y1 = torch.zeros((2, 8), dtype=torch.float32, device="cuda")
    y2 = torch.zeros((2, 8), dtype=torch.float32, device="cuda")
    for L, bl in ((L2, b2), (L3, b3)):
        with pytest.raises(N.BitcosError) as e:
            api.Batch([L1, L], [dev(b1), dev(bl)], [x, x], [y1, y2])
        assert e.value.status == N.E_UNSUPPORTED


# ---------------------------------------------------------------------------
# Full configured size: the Qwen3-32B-like layer set at batch 4 and 16
# ---------------------------------------------------------------------------

@functools.lru_cache(maxsize=1)
def _qwen32_matrix(midx):
    wk = wl.WORKLOADS["qwen3_32b_layers"]
    return wl.matrix_inputs(wk.cid, 0, midx, wk.matrices[midx])


@pytest.mark.parametrize("m", [4, 16])
@pytest.mark.parametrize("midx", [0, 1, 4, 6])
def test_full_size_qwen3_32b_small_batch(midx, m):
    wk = wl.WORKLOADS["qwen3_32b_layers"]
    spec = wk.matrices[midx]
    w, sc = _qwen32_matrix(midx)
    rows = sampled_rows(spec.n, 48, midx)
    scr = sc.reshape(spec.n, -1)[rows].reshape(-1)
    xb = wl.activation_inputs(wk.cid, "bf16", m, spec.k)
    y, _ = run(N.FMT_BITCOS, w, sc, 128, xb, "bf16")
    check_bf16(y[:, rows], O.dense_gemv(w[rows], scr, 128, xb, x_is_bf16_bits=True),
               bf16_bound(w[rows], scr, 128, xb))
    x = wl.activation_inputs(wk.cid, "int8", m, spec.k)
    y, _ = run(N.FMT_BITCOS, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW)
    assert np.array_equal(y[:, rows], O.dense_gemv_raw(w[rows], x).astype(np.int32))


def test_qwen3_32b_layer_in_one_small_batch_launch():
    """All seven matrices of a Qwen3-32B-like layer (K = 5120 and 25600) in one
    batch table at M = 4: the launch splits its steps (not its 32-row units)
    over the waves, so waves start inside units and GEMVs of both row
    lengths; every GEMV must still match the oracle on sampled rows, twice."""
    wk = wl.WORKLOADS["qwen3_32b_layers"]
    m = 4
    mats = [wl.matrix_inputs(wk.cid, 1, i, spec) for i, spec in enumerate(wk.matrices)]
    for kind in ("int8", "bf16"):
        layouts, blobs, xs, ys, xsrc = [], [], [], [], []
        for i, (spec, (w, sc)) in enumerate(zip(wk.matrices, mats)):
            L, blob = api.plan_and_pack(N.FMT_BITCOS, w, sc, 128)
            x = wl.activation_inputs(wk.cid, kind, m, spec.k, salt=i)
            layouts.append(L)
            blobs.append(torch.from_numpy(blob).cuda())
            xs.append(to_dev_x(x, kind))
            xsrc.append(x)
            ys.append(torch.full((m, spec.n), -7.0, dtype=torch.float32, device="cuda"))
        say("qwen3-32b layer, one small-batch launch", kind)
        ymode = N.Y_I32_RAW if kind == "int8" else N.Y_F32
        if kind == "int8":
            ys = [torch.full((m, spec.n), -7, dtype=torch.int32, device="cuda") for spec in wk.matrices]
        b = api.Batch(layouts, blobs, xs, ys, y_mode=ymode)
        assert b.m == m
        first = None
        for rep in range(2):
            b.run()
            torch.cuda.synchronize()
            got = [y.cpu().numpy() for y in ys]
            for i, (spec, (w, sc), x, g) in enumerate(zip(wk.matrices, mats, xsrc, got)):
                rows = sampled_rows(spec.n, 24, 70 + i)
                if kind == "int8":
                    assert np.array_equal(g[:, rows], O.dense_gemv_raw(w[rows], x).astype(np.int32)), spec.name
                else:
                    scr = sc.reshape(spec.n, -1)[rows].reshape(-1)
                    check_bf16(g[:, rows], O.dense_gemv(w[rows], scr, 128, x, x_is_bf16_bits=True),
                               bf16_bound(w[rows], scr, 128, x))
            if first is None:
                first = [g.copy() for g in got]
            else:
                for g, f in zip(got, first):
                    assert np.array_equal(g.view(np.uint32), f.view(np.uint32))
