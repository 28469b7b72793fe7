"""GPU parity of the accumulating output modes (BITCOS_Y_F32_ADD,
BITCOS_Y_I32_RAW_ADD): y += (S (.) W) x on every kernel, and a matrix stored
as column blocks (a split of K) whose block GEMVs add into one output.

The added quantity is the same dense definition as the plain modes (Sec.
II-C); the bars are those of parity_checks.py applied to y - y0, where y0 is
what y held before the call (the fp32 addition itself rounds once more, so
the fp32 cases allow one extra rounding of |y|).  Raw int32 sums are exact:
y == y0 + sum_k W x bit for bit.
"""

import numpy as np
import pytest

import oracle as O
import workloads as wl
from parity_checks import bf16_bound, group_bound, inputs, say, to_dev_x

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2609_16338_amd import _native as N  # noqa: E402
from paper_2609_16338_amd import api  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    N.lib()


FMTS = {"bitcos": N.FMT_BITCOS, "trit5": N.FMT_TRIT5, "bit2": N.FMT_BIT2}


def _run_add(fmt, w, sc, group, x, kind, xscale=None, raw=False, unit=0, m=1):
    L, blob = api.plan_and_pack(fmt, w, sc, group, unit)
    bd = torch.from_numpy(blob).cuda()
    xd = to_dev_x(x, kind)
    n = w.shape[0]
    rng = np.random.default_rng(n * 7 + w.shape[1])
    if raw:
        y0 = rng.integers(-1000, 1000, size=(m, n)).astype(np.int32)
    else:
        y0 = rng.standard_normal((m, n)).astype(np.float32)
    y = torch.from_numpy(y0.copy()).cuda()
    xs = None if xscale is None else torch.from_numpy(np.ascontiguousarray(xscale, np.float32)).cuda()
    api.gemv(L, bd, xd, y, xs, N.Y_I32_RAW_ADD if raw else N.Y_F32_ADD)
    torch.cuda.synchronize()
    return y0, y.cpu().numpy(), L


@pytest.mark.parametrize("fmt", list(FMTS))
@pytest.mark.parametrize("case", ["per_tensor_bf16", "grouped_bf16", "grouped_int8_xscale", "raw_int8"])
def test_single_call_adds(fmt, case):
    n, k = 77, 2560
    group = 0 if case == "per_tensor_bf16" else 128
    w, sc = inputs(n, k, 0.42, group, 31)
    say("add", fmt, case)
    if case.endswith("bf16"):
        xb = wl.act_bf16(1, k, wl.rng_for(310, k))
        y0, y, _ = _run_add(FMTS[fmt], w, sc, group, xb, "bf16")
        ref = O.dense_gemv(w, sc, group, xb, x_is_bf16_bits=True).astype(np.float64)
        bar = 1e-3 * bf16_bound(w, sc, group, xb) + 2 ** -23 * np.abs(y.astype(np.float64))
    elif case == "grouped_int8_xscale":
        q, a = O.quantize_activations(wl.act_bf16(1, k, wl.rng_for(311, k)))
        y0, y, _ = _run_add(FMTS[fmt], w, sc, group, q, "int8", xscale=a)
        ref = O.dense_gemv(w, sc, group, q, a).astype(np.float64)
        bar = 1e-5 * group_bound(w, sc, group, q, a) + 2 ** -23 * np.abs(y.astype(np.float64))
    else:
        x = wl.act_int8(1, k, wl.rng_for(312, k))
        y0, y, _ = _run_add(FMTS[fmt], w, sc, group, x, "int8", raw=True)
        assert np.array_equal(y, y0 + O.dense_gemv_raw(w, x).astype(np.int32))
        return
    err = np.abs(y.astype(np.float64) - (y0.astype(np.float64) + ref))
    assert np.all(err <= bar), float((err / bar).max())


@pytest.mark.parametrize("k", [256, 6912])
def test_add_on_the_general_and_small_batch_kernels(k):
    """unit_rows = 3 (general kernel) and m = 4 (small-batch kernel)."""
    n = 50
    w, sc = inputs(n, k, 0.45, 128, 32)
    x = wl.act_int8(1, k, wl.rng_for(320, k))
    y0, y, L = _run_add(N.FMT_BITCOS, w, sc, 128, x, "int8", raw=True, unit=3)
    assert api.describe(L, 1, N.X_I8).kernel == N.KERNEL_GENERAL
    assert np.array_equal(y, y0 + O.dense_gemv_raw(w, x).astype(np.int32))
    xb = wl.act_bf16(4, k, wl.rng_for(321, k))
    y0, y, L = _run_add(N.FMT_BITCOS, w, sc, 128, xb, "bf16", m=4)
    assert api.describe(L, 4, N.X_BF16).kernel == N.KERNEL_SMALL_BATCH
    ref = O.dense_gemv(w, sc, 128, xb, x_is_bf16_bits=True).astype(np.float64)
    bar = 1e-3 * bf16_bound(w, sc, 128, xb) + 2 ** -23 * np.abs(y.astype(np.float64))
    assert np.all(np.abs(y - (y0 + ref)) <= bar)


@pytest.mark.parametrize("kind", ["bf16", "int8"])
@pytest.mark.parametrize("fmt", list(FMTS))
def test_column_blocks_add_up_to_the_whole_row(kind, fmt):
    """A 25600-wide matrix stored as five 5120-wide column blocks: block 0
    writes y, blocks 1..4 add onto it, in stream order; y is the GEMV of the
    whole matrix (and the same bits on a second run)."""
    n, k, kb = 300, 25600, 5120
    w, sc = inputs(n, k, 0.45, 128, 33, lo=0.005, hi=0.05)
    if kind == "bf16":
        x = wl.act_bf16(1, k, wl.rng_for(330))
        a = None
        ref = O.dense_gemv(w, sc, 128, x, x_is_bf16_bits=True).astype(np.float64)
        bar = 1e-3 * bf16_bound(w, sc, 128, x)
    else:
        x, a = O.quantize_activations(wl.act_bf16(1, k, wl.rng_for(331)))
        ref = O.dense_gemv(w, sc, 128, x, a).astype(np.float64)
        bar = 1e-5 * group_bound(w, sc, 128, x, a)
    scg = sc.reshape(n, k // 128)
    blocks = []
    for k0 in range(0, k, kb):
        wb = np.ascontiguousarray(w[:, k0:k0 + kb])
        sb = np.ascontiguousarray(scg[:, k0 // 128:(k0 + kb) // 128]).reshape(-1)
        L, blob = api.plan_and_pack(FMTS[fmt], wb, sb, 128)
        xb = to_dev_x(np.ascontiguousarray(x[:, k0:k0 + kb]), kind)
        xsb = None if a is None else torch.from_numpy(np.ascontiguousarray(a[:, k0 // 128:(k0 + kb) // 128])).cuda()
        blocks.append((L, torch.from_numpy(blob).cuda(), xb, xsb))
    say("column blocks", fmt, kind)
    outs = []
    for _ in range(2):
        y = torch.full((1, n), float("nan"), dtype=torch.float32, device="cuda")
        for c, (L, bd, xb, xsb) in enumerate(blocks):
            api.gemv(L, bd, xb, y, xsb, N.Y_F32 if c == 0 else N.Y_F32_ADD)
        torch.cuda.synchronize()
        outs.append(y.cpu().numpy())
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
    err = np.abs(outs[0].astype(np.float64) - ref)
    assert np.all(err <= bar + 1e-30), float((err / (bar + 1e-30)).max())
    # The same blocks with blocks 1..4 written to a partial buffer and added by
    # bitcos_add_partials: the same fp32 additions in the same order, so the
    # same bits as the accumulating mode.
    y = torch.full((1, n), float("nan"), dtype=torch.float32, device="cuda")
    parts = torch.full((len(blocks) - 1, 1, n), float("nan"), dtype=torch.float32, device="cuda")
    for c, (L, bd, xb, xsb) in enumerate(blocks):
        api.gemv(L, bd, xb, y if c == 0 else parts[c - 1], xsb, N.Y_F32)
    api.add_partials(y, parts)
    torch.cuda.synchronize()
    assert np.array_equal(y.cpu().numpy().view(np.uint32), outs[0].view(np.uint32))


@pytest.mark.parametrize("n,nparts,offset", [(1, 1, 0), (7, 3, 0), (4096, 4, 0), (4096, 2, 1), (1000003, 4, 0),
                                             (3 * 5120 * 64, 4, 0)])
def test_add_partials_is_the_sum_in_block_order(n, nparts, offset):
    """bitcos_add_partials: y[i] + parts[0][i] + ... + parts[P-1][i], one fp32
    addition per part, left to right -- against the same additions in numpy,
    bit-exact; four elements per thread on aligned buffers of a multiple of 4
    elements, one otherwise (offset 1 misaligns both buffers)."""
    rng = np.random.default_rng(n + nparts)
    y0 = rng.standard_normal(n + offset).astype(np.float32)
    p0 = rng.standard_normal((nparts, n + offset)).astype(np.float32)
    ref = y0[offset:].copy()
    for j in range(nparts):
        ref = (ref + p0[j, offset:]).astype(np.float32)
    yb = torch.from_numpy(y0).cuda()
    pb = torch.from_numpy(p0.reshape(-1)).cuda()
    y = yb[offset:]
    if offset:
        # parts as one buffer of nparts * n elements starting one element in
        parts = torch.from_numpy(np.ascontiguousarray(p0[:, offset:]).reshape(-1))
        pb = torch.empty(nparts * n + 1, dtype=torch.float32, device="cuda")
        pb[1:].copy_(parts.cuda())
        pview = pb[1:].view(nparts, n)
    else:
        pview = pb.view(nparts, n + offset)
    say("add_partials", n, nparts, offset)
    api.add_partials(y, pview)
    torch.cuda.synchronize()
    assert np.array_equal(y.cpu().numpy().view(np.uint32), ref.view(np.uint32))


def test_add_modes_in_batch_tables():
    """A batch table in an _ADD mode adds every GEMV's result onto its y."""
    k = 2560
    specs = [(64, 0.42), (5, 0.0), (300, 0.5)]
    layouts, blobs, xs, ys, y0s, refs = [], [], [], [], [], []
    for i, (n, z) in enumerate(specs):
        w, sc = inputs(n, k, z, 0, 340 + i)
        x = wl.act_int8(1, k, wl.rng_for(341, i))
        L, blob = api.plan_and_pack(N.FMT_BITCOS, w, sc, 0)
        y0 = np.random.default_rng(i).integers(-50, 50, size=n).astype(np.int32)
        layouts.append(L)
        blobs.append(torch.from_numpy(blob).cuda())
        xs.append(torch.from_numpy(x.reshape(-1)).cuda())
        ys.append(torch.from_numpy(y0.copy()).cuda())
        y0s.append(y0)
        refs.append(O.dense_gemv_raw(w, x).astype(np.int32).reshape(-1))
    b = api.Batch(layouts, blobs, xs, ys, None, y_mode=N.Y_I32_RAW_ADD)
    b.run()
    torch.cuda.synchronize()
    for y, y0, ref in zip(ys, y0s, refs):
        assert np.array_equal(y.cpu().numpy(), y0 + ref)


def test_add_mode_argument_checks():
    w, sc = inputs(8, 256, 0.4, 128, 35)
    L, blob = api.plan_and_pack(N.FMT_BITCOS, w, sc, 128)
    bd = torch.from_numpy(blob).cuda()
    xb = to_dev_x(wl.act_bf16(1, 256, wl.rng_for(350)), "bf16")
    y = torch.zeros((1, 8), dtype=torch.int32, device="cuda")
    st = N.lib().bitcos_gemv(L, bd.data_ptr(), 1, xb.data_ptr(), N.X_BF16, None, y.data_ptr(),
                             N.Y_I32_RAW_ADD, None)  # raw sums need int8 activations
    assert st == N.E_ARG
    st = N.lib().bitcos_gemv(L, bd.data_ptr(), 1, xb.data_ptr(), N.X_BF16, None, y.data_ptr(), 5, None)
    assert st == N.E_ARG
