"""GPU parity of the batch-1 BITCOS path for group- and activation-scaled
layouts (the streaming kernel), and repeatability of every batch-1 kernel.

Group scales multiply each 128-weight group's sum (Sec. II-C); a lane's words
start at every phase of a group of four words across the tile widths below,
so words cross into the next scale group at every position.  Bars as in
test_gpu_parity.py: group- or activation-scaled int8 within 1e-5 of
sum |S a A|, raw int32 sums bit-exact, bf16 within 1e-3 of sum |S W x| per
element and in norm.

The repeatability test runs each case ten times and requires identical bits:
the kernels stage each step's sign block into LDS with LDS-DMA and must not
read it before it has landed (a read too early gives stale signs, wrong rows
and run-to-run differences).
"""

import numpy as np
import pytest

import oracle as O
import workloads as wl
from parity_checks import bf16_bound, check_bf16, check_grouped, group_bound, inputs, run, say, to_dev_x

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
api = pytest.importorskip("paper_2609_16338_amd.api")
from paper_2609_16338_amd import _native as N  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    N.lib()


# K -> (words per lane, lanes per row): 128 (1, 4), 256 (2, 4), 384 (3, 4),
# 640 (5, 4), 1024 (8, 4), 1152 (5, 8) ragged, 2048 (8, 8), 2560 (5, 16),
# 4096 (8, 16), 5120 (5, 32), 6912 (7, 32) ragged, 8192 (8, 32), 12288 (6, 64)
# (int8; bf16: 1024 (4, 8), 2048 (4, 16), 4096 (4, 32), 8192 (4, 64)).
KS = [128, 256, 384, 640, 1024, 1152, 2048, 2560, 4096, 5120, 6912, 8192, 12288]


def _kernel(L, kind):
    return api.describe(L, 1, N.X_I8 if kind == "int8" else N.X_BF16).kernel


@pytest.mark.parametrize("k", KS)
def test_int8_group_and_activation_scales(k):
    n = 45
    w, sc = inputs(n, k, 0.42, 128, 16, lo=0.005, hi=0.05)
    x = wl.act_int8(1, k, wl.rng_for(116, k))
    y, L = run(N.FMT_BITCOS, w, sc, 128, x, "int8")
    assert _kernel(L, "int8") == N.KERNEL_STREAMING
    check_grouped(y, O.dense_gemv(w, sc, 128, x), group_bound(w, sc, 128, x))
    # per-group activation scales, with group scales and with one scale per tensor
    q, a = O.quantize_activations(wl.act_bf16(1, k, wl.rng_for(117, k)))
    y, _ = run(N.FMT_BITCOS, w, sc, 128, q, "int8", xscale=a)
    check_grouped(y, O.dense_gemv(w, sc, 128, q, a), group_bound(w, sc, 128, q, a))
    w1, s1 = inputs(n, k, 0.42, 0, 17)
    y, _ = run(N.FMT_BITCOS, w1, s1, 0, q, "int8", xscale=a)
    check_grouped(y, O.dense_gemv(w1, s1, 0, q, a), group_bound(w1, s1, 0, q, a))
    # raw sums ignore every scale and stay bit-exact
    y, _ = run(N.FMT_BITCOS, w, sc, 128, q, "int8", xscale=a, y_mode=N.Y_I32_RAW)
    assert np.array_equal(y, O.dense_gemv_raw(w, q).astype(np.int32))


@pytest.mark.parametrize("k", KS)
def test_bf16_group_scales(k):
    n = 39
    w, sc = inputs(n, k, 0.467, 128, 18, lo=0.005, hi=0.05)
    xb = wl.act_bf16(1, k, wl.rng_for(118, k))
    y, L = run(N.FMT_BITCOS, w, sc, 128, xb, "bf16")
    assert _kernel(L, "bf16") == N.KERNEL_STREAMING
    check_bf16(y, O.dense_gemv(w, sc, 128, xb, x_is_bf16_bits=True), bf16_bound(w, sc, 128, xb))


@pytest.mark.parametrize("k", [256, 2560, 6912])
@pytest.mark.parametrize("z", [0.0, 1.0])
def test_grouped_degenerate_densities(k, z):
    n = 21
    w, sc = inputs(n, k, z, 128, 19)
    q, a = O.quantize_activations(wl.act_bf16(1, k, wl.rng_for(119, k)))
    y, _ = run(N.FMT_BITCOS, w, sc, 128, q, "int8", xscale=a)
    check_grouped(y, O.dense_gemv(w, sc, 128, q, a), group_bound(w, sc, 128, q, a))
    xb = wl.act_bf16(1, k, wl.rng_for(120, k))
    y, _ = run(N.FMT_BITCOS, w, sc, 128, xb, "bf16")
    check_bf16(y, O.dense_gemv(w, sc, 128, xb, x_is_bf16_bits=True), bf16_bound(w, sc, 128, xb))


@pytest.mark.parametrize("k", [2560, 6912])
def test_bf16_with_activation_scales(k):
    """bf16 activations with per-group activation scales: y = sum_g S a A."""
    n = 23
    w, sc = inputs(n, k, 0.42, 128, 20)
    xb = wl.act_bf16(1, k, wl.rng_for(121, k))
    a = wl.rng_for(122, k).uniform(0.5, 2.0, size=(1, k // 128)).astype(np.float32)
    y, _ = run(N.FMT_BITCOS, w, sc, 128, xb, "bf16", xscale=a)
    ref = O.dense_gemv(w, sc, 128, xb, a, x_is_bf16_bits=True)
    check_bf16(y, ref, bf16_bound(w, sc, 128, xb) * float(a.max()))


@pytest.mark.parametrize("k", [256, 2560, 6912, 8192])
@pytest.mark.parametrize("kind", ["int8", "bf16"])
def test_grouped_batch_tables(k, kind):
    """Grouped GEMVs of one tile in one launch (int8 with activation scales), twice: same bits."""
    specs = [(64, 0.42), (5, 0.0), (300, 0.5), (33, 1.0), (129, 0.467)]
    layouts, blobs, xs, xss, ys, refs, bounds = [], [], [], [], [], [], []
    for i, (n, z) in enumerate(specs):
        w, sc = inputs(n, k, z, 128, 600 + i)
        if kind == "int8":
            x, a = O.quantize_activations(wl.act_bf16(1, k, wl.rng_for(601, i, k)))
            refs.append(O.dense_gemv(w, sc, 128, x, a))
            bounds.append(group_bound(w, sc, 128, x, a))
            xss.append(torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda())
        else:
            x = wl.act_bf16(1, k, wl.rng_for(602, i, k))
            refs.append(O.dense_gemv(w, sc, 128, x, x_is_bf16_bits=True))
            bounds.append(bf16_bound(w, sc, 128, x))
        L, blob = api.plan_and_pack(N.FMT_BITCOS, w, sc, 128)
        layouts.append(L)
        blobs.append(torch.from_numpy(blob).cuda())
        xs.append(to_dev_x(x, kind).reshape(-1))
        ys.append(torch.full((n,), -7.0, dtype=torch.float32, device="cuda"))
    say("grouped batch", k, kind)
    b = api.Batch(layouts, blobs, xs, ys, xss if kind == "int8" else None)
    first = None
    for rep in range(2):
        b.run()
        torch.cuda.synchronize()
        got = [y.cpu().numpy()[None] for y in ys]
        for g, ref, bound in zip(got, refs, bounds):
            if kind == "int8":
                check_grouped(g, ref, bound)
            else:
                check_bf16(g, ref, bound)
        if first is None:
            first = [g.copy() for g in got]
        else:
            for g, f in zip(got, first):
                assert np.array_equal(g.view(np.uint32), f.view(np.uint32))


@pytest.mark.parametrize("k", [1024, 2560, 4096, 6912, 12288])
@pytest.mark.parametrize("group", [0, 128])
def test_repeated_runs_identical(k, group):
    """Ten runs of each batch-1 kernel (matrix cores: one scale per tensor;
    streaming: group scales), int8 and bf16: every run within the bar and
    bit-identical to the first."""
    n = 45
    w, sc = inputs(n, k, 0.42, group, 700 + k)
    x = wl.act_int8(1, k, wl.rng_for(701, k))
    xb = wl.act_bf16(1, k, wl.rng_for(702, k))
    ref8 = O.dense_gemv(w, sc, group, x)
    b8 = group_bound(w, sc, group, x)
    refb = O.dense_gemv(w, sc, group, xb, x_is_bf16_bits=True)
    bb = bf16_bound(w, sc, group, xb)
    L, blob = api.plan_and_pack(N.FMT_BITCOS, w, sc, group)
    say("repeat", k, f"group={group}", f"kernel={_kernel(L, 'int8')}")
    blob_d = torch.from_numpy(blob).cuda()
    for kind, xv, ref in (("int8", x, ref8), ("bf16", xb, refb)):
        xd = to_dev_x(xv, kind)
        first = None
        for rep in range(10):
            y = torch.full((1, n), -7.0, dtype=torch.float32, device="cuda")
            api.gemv(L, blob_d, xd, y)
            torch.cuda.synchronize()
            got = y.cpu().numpy()
            if kind == "int8":
                if group == 0:
                    assert np.array_equal(got, ref)
                else:
                    check_grouped(got, ref, b8)
            else:
                check_bf16(got, ref, bb)
            if first is None:
                first = got.copy()
            else:
                assert np.array_equal(got.view(np.uint32), first.view(np.uint32)), (kind, rep)


# Batch-1 rows longer than every batch-1 tile: bf16 K > 16384 (a lane's
# activations no longer fit its registers), int8 K > 32768.  They run the
# small-batch kernel with one activation row.
@pytest.mark.parametrize("k,kind,group", [(16512, "bf16", 128), (25600, "bf16", 0), (25600, "bf16", 128),
                                          (32896, "int8", 0), (32896, "int8", 128)])
def test_batch1_long_rows(k, kind, group):
    n = 37
    w, sc = inputs(n, k, 0.45, group, 30, lo=0.005, hi=0.05)
    if kind == "bf16":
        xb = wl.act_bf16(1, k, wl.rng_for(130, k))
        y, L = run(N.FMT_BITCOS, w, sc, group, xb, "bf16")
        assert _kernel(L, "bf16") == N.KERNEL_SMALL_BATCH
        check_bf16(y, O.dense_gemv(w, sc, group, xb, x_is_bf16_bits=True), bf16_bound(w, sc, group, xb))
        return
    x = wl.act_int8(1, k, wl.rng_for(131, k))
    y, L = run(N.FMT_BITCOS, w, sc, group, x, "int8")
    assert _kernel(L, "int8") == N.KERNEL_SMALL_BATCH
    if group == 0:
        assert np.array_equal(y, O.dense_gemv(w, sc, 0, x))
    else:
        check_grouped(y, O.dense_gemv(w, sc, group, x), group_bound(w, sc, group, x))
    y, _ = run(N.FMT_BITCOS, w, sc, group, x, "int8", y_mode=N.Y_I32_RAW)
    assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32))
    q, a = O.quantize_activations(wl.act_bf16(1, k, wl.rng_for(132, k)))
    y, _ = run(N.FMT_BITCOS, w, sc, group, q, "int8", xscale=a)
    check_grouped(y, O.dense_gemv(w, sc, group, q, a), group_bound(w, sc, group, q, a))


def test_batch1_long_rows_batch_table():
    """Long-row GEMVs of one batch (m = 1, the small-batch kernel), twice: same bits."""
    k = 25600
    specs = [(48, 0.45), (5, 0.0), (131, 0.6)]
    layouts, blobs, xs, ys, refs, bounds = [], [], [], [], [], []
    for i, (n, z) in enumerate(specs):
        w, sc = inputs(n, k, z, 128, 800 + i, lo=0.005, hi=0.05)
        x = wl.act_bf16(1, k, wl.rng_for(801, i))
        refs.append(O.dense_gemv(w, sc, 128, x, x_is_bf16_bits=True))
        bounds.append(bf16_bound(w, sc, 128, x))
        L, blob = api.plan_and_pack(N.FMT_BITCOS, w, sc, 128)
        assert _kernel(L, "bf16") == N.KERNEL_SMALL_BATCH
        layouts.append(L)
        blobs.append(torch.from_numpy(blob).cuda())
        xs.append(to_dev_x(x, "bf16").reshape(-1))
        ys.append(torch.full((n,), -7.0, dtype=torch.float32, device="cuda"))
    say("long-row batch", k)
    b = api.Batch(layouts, blobs, xs, ys)
    first = None
    for rep in range(2):
        b.run()
        torch.cuda.synchronize()
        got = [y.cpu().numpy()[None] for y in ys]
        for g, ref, bound in zip(got, refs, bounds):
            check_bf16(g, ref, bound)
        if first is None:
            first = [g.copy() for g in got]
        else:
            for g, f in zip(got, first):
                assert np.array_equal(g.view(np.uint32), f.view(np.uint32))
