"""GPU parity: the HIP GEMVs of libbitcos against the CPU oracle.

Every case packs W with the library (byte-identical to the oracle's packing,
see test_host_lib.py), runs the kernel on cuda:0 through the C ABI and
compares with the oracle's dense definition on the same seeded inputs.

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
import pytest

import oracle as O
import workloads as wl
from parity_checks import (bf16_bound, check_bf16, check_grouped, group_bound, inputs, run, sampled_rows as _sampled,
                           say, to_dev_x)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
api = pytest.importorskip("paper_2609_16338_amd.api")
from paper_2609_16338_amd import _native as N  # noqa: E402

FMTS = [N.FMT_BITCOS, N.FMT_TRIT5, N.FMT_BIT2]
FMT_NAME = {N.FMT_BITCOS: "bitcos", N.FMT_TRIT5: "trit5", N.FMT_BIT2: "bit2"}


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    N.lib()


# ---------------------------------------------------------------------------
# The smallest configured instance
# ---------------------------------------------------------------------------

def test_single_256x1024_int8():
    spec = wl.WORKLOADS["single_256x1024"].matrices[0]
    w, sc = wl.matrix_inputs(1, 0, 0, spec)
    x = wl.activation_inputs(1, "int8", 1, spec.k)
    for fmt in FMTS:
        y, L = run(fmt, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW)
        assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32))
        y, L = run(fmt, w, sc, 128, x, "int8")
        check_grouped(y, O.dense_gemv(w, sc, 128, x), group_bound(w, sc, 128, x))
    Lb = api.bitcos_plan(w, 128, 0)
    zeros = int(np.count_nonzero(w == 0))
    assert Lb.payload_bits == 2 * 256 * 1024 - zeros + 256 * 8 * 16   # (2 - z + 1/8) * N * K


# ---------------------------------------------------------------------------
# Shapes of every configured layer, ragged row counts, all three formats
# ---------------------------------------------------------------------------

KS = [128, 256, 1024, 2560, 4096, 5120, 6912, 8192, 12288, 25600]


@pytest.mark.parametrize("k", KS)
def test_raw_int32_exact_all_formats(k):
    n = 37 if k <= 8192 else 19
    w, sc = inputs(n, k, 0.42, 128, 1)
    x = wl.act_int8(1, k, wl.rng_for(92, k))
    ref = O.dense_gemv_raw(w, x).astype(np.int32)
    for fmt in FMTS:
        y, _ = run(fmt, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW)
        assert np.array_equal(y, ref), FMT_NAME[fmt]


@pytest.mark.parametrize("k", KS)
def test_group_scaled_int8_all_formats(k):
    n = 29
    w, sc = inputs(n, k, 0.467, 128, 2, 0.005, 0.05)
    x = wl.act_int8(1, k, wl.rng_for(93, k))
    ref = O.dense_gemv(w, sc, 128, x)
    bound = group_bound(w, sc, 128, x)
    for fmt in FMTS:
        y, _ = run(fmt, w, sc, 128, x, "int8")
        check_grouped(y, ref, bound)


@pytest.mark.parametrize("k", [256, 2560, 6912])
def test_per_tensor_int8_bit_exact(k):
    n = 41
    w, sc = inputs(n, k, 0.42, 0, 3)
    x = wl.act_int8(1, k, wl.rng_for(94, k))
    ref = O.dense_gemv(w, sc, 0, x)
    for fmt in FMTS:
        y, _ = run(fmt, w, sc, 0, x, "int8")
        assert np.array_equal(y, ref), FMT_NAME[fmt]


def test_per_tensor_k_multiple_of_32_bitcos():
    w, sc = inputs(9, 96, 0.4, 0, 4)
    x = wl.act_int8(1, 96, wl.rng_for(95))
    y, _ = run(N.FMT_BITCOS, w, sc, 0, x, "int8", y_mode=N.Y_I32_RAW)
    assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32))
    y, _ = run(N.FMT_BITCOS, w, sc, 0, x, "int8")
    assert np.array_equal(y, O.dense_gemv(w, sc, 0, x))


BF16_KS = [128, 1024, 2560, 4096, 5120, 6912, 8192, 12288]


@pytest.mark.parametrize("k", BF16_KS)
@pytest.mark.parametrize("group", [0, 128])
def test_bf16_all_formats(k, group):
    n = 23
    w, sc = inputs(n, k, 0.42, group, 5)
    xb = wl.act_bf16(1, k, wl.rng_for(96, k))
    ref = O.dense_gemv(w, sc, group, xb, x_is_bf16_bits=True)
    bound = bf16_bound(w, sc, group, xb)
    for fmt in FMTS:
        y, _ = run(fmt, w, sc, group, xb, "bf16")
        check_bf16(y, ref, bound)


@pytest.mark.parametrize("k", [2560, 5120])
@pytest.mark.parametrize("kind", ["bf16", "int8"])
def test_trit5_twenty_lane_segments_multi_step(kind, k):
    """Five-trit on rows of 20 or 40 blocks runs 20-lane segments: three rows
    per wave step, the row's partial sums moved by ds_bpermute rounds, the
    last four lanes idle.  One GEMV with more steps than twice the most waves
    the GPU holds, so every wave of the persistent grid takes several; the row
    count leaves the last step one row short.  Sampled rows (and the first and
    last) against the oracle (int8: raw int32 sums, bit-exact); two runs give
    identical bits."""
    from parity_checks import sampled_rows
    p = torch.cuda.get_device_properties(0)
    resident = p.multi_processor_count * max(p.max_threads_per_multi_processor // 64, 1)
    n = 3 * 2 * resident + 2
    w, sc = inputs(n, k, 0.42, 128, 78)
    if kind == "bf16":
        x = wl.act_bf16(1, k, wl.rng_for(98, k))
        xd = torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda().reshape(-1)
    else:
        x = wl.act_int8(1, k, wl.rng_for(99, k))
        xd = torch.from_numpy(x).cuda().reshape(-1)
    L, blob = api.plan_and_pack(N.FMT_TRIT5, w, sc, 128)
    info = api.describe(L, 1, N.X_BF16 if kind == "bf16" else N.X_I8)
    assert (info.seg_lanes, info.rows_per_step, info.per_lane) == (20, 3, k // 2560)
    assert info.waves > 2 * resident
    say("trit5 20-lane", kind, n, k, info.waves)
    blob_d = torch.from_numpy(blob).cuda()
    y_mode = N.Y_F32 if kind == "bf16" else N.Y_I32_RAW
    outs = []
    for _ in range(2):
        if kind == "bf16":
            y = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
        else:
            y = torch.full((n,), -7, dtype=torch.int32, device="cuda")
        api.gemv(L, blob_d, xd, y, None, y_mode)
        torch.cuda.synchronize()
        outs.append(y.cpu().numpy())
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
    rows = sampled_rows(n, 300, k)
    if kind == "int8":
        assert np.array_equal(outs[0][rows].astype(np.int64), O.dense_gemv_raw(w[rows], x)[0])
        return
    assert np.all(np.isfinite(outs[0]))
    scr = sc.reshape(n, -1)[rows].reshape(-1)
    ref = O.dense_gemv(w[rows], scr, 128, x, x_is_bf16_bits=True)
    check_bf16(outs[0][rows][None], ref, bf16_bound(w[rows], scr, 128, x))


def test_bf16_unsupported_shape_is_an_error_not_a_fallback():
    # Rows too long for the batch-1 tiles with two rows per sign offset: the
    # small-batch kernel needs one offset per row, so no kernel takes it.
    w, sc = inputs(3, 25600, 0.42, 128, 6)
    xb = wl.act_bf16(1, 25600, wl.rng_for(97))
    with pytest.raises(N.BitcosError) as e:
        run(N.FMT_BITCOS, w, sc, 128, xb, "bf16", unit=2)
    assert e.value.status == N.E_UNSUPPORTED


@pytest.mark.parametrize("group", [0, 128])
def test_int8_with_activation_scales(group):
    # The int8-quantised variant of bf16 activations (per group of 128).
    k, n = 2560, 33
    w, sc = inputs(n, k, 0.42, group, 7)
    xb = wl.act_bf16(1, k, wl.rng_for(98))
    q, a = O.quantize_activations(xb)
    ref = O.dense_gemv(w, sc, group, q, a)
    bound = group_bound(w, sc, group, q, a)
    for fmt in FMTS:
        y, _ = run(fmt, w, sc, group, q, "int8", xscale=a)
        check_grouped(y, ref, bound)


# ---------------------------------------------------------------------------
# Edge cases
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("z", [0.0, 1.0])
def test_degenerate_densities(z):
    w, sc = inputs(17, 1024, z, 128, 8)
    x = wl.act_int8(1, 1024, wl.rng_for(99))
    for fmt in FMTS:
        y, _ = run(fmt, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW)
        assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32))


def test_single_row_and_single_group():
    w, sc = inputs(1, 128, 0.3, 128, 9)
    x = wl.act_int8(1, 128, wl.rng_for(100))
    xb = wl.act_bf16(1, 128, wl.rng_for(101))
    for fmt in FMTS:
        y, _ = run(fmt, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW)
        assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32))
        y, _ = run(fmt, w, sc, 128, xb, "bf16")
        check_bf16(y, O.dense_gemv(w, sc, 128, xb, x_is_bf16_bits=True), bf16_bound(w, sc, 128, xb))


@pytest.mark.parametrize("unit", [1, 2, 5, 7, 1000])
def test_bitcos_unit_rows_variants(unit):
    w, sc = inputs(45, 2560, 0.45, 128, 10)
    w[3] = 0
    w[10, :] = -1
    x = wl.act_int8(1, 2560, wl.rng_for(102))
    y, L = run(N.FMT_BITCOS, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW, unit=unit)
    assert L.unit_rows == unit
    assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32))
    xb = wl.act_bf16(1, 2560, wl.rng_for(103))
    y, _ = run(N.FMT_BITCOS, w, sc, 128, xb, "bf16", unit=unit)
    check_bf16(y, O.dense_gemv(w, sc, 128, xb, x_is_bf16_bits=True), bf16_bound(w, sc, 128, xb))


def test_extreme_activations():
    k = 1024
    w, sc = inputs(19, k, 0.2, 128, 11)
    x = np.full((1, k), -127, np.int8)
    x[0, ::3] = 127
    for fmt in FMTS:
        y, _ = run(fmt, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW)
        assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32))


def test_deterministic_repeat():
    w, sc = inputs(300, 6912, 0.42, 128, 12)
    x = wl.act_int8(1, 6912, wl.rng_for(104))
    xb = wl.act_bf16(1, 6912, wl.rng_for(105))
    for fmt in FMTS:
        a, _ = run(fmt, w, sc, 128, x, "int8")
        b, _ = run(fmt, w, sc, 128, x, "int8")
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
        a, _ = run(fmt, w, sc, 128, xb, "bf16")
        b, _ = run(fmt, w, sc, 128, xb, "bf16")
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


# ---------------------------------------------------------------------------
# Full configured sizes, checked on sampled rows (the launch bench.py times)
# ---------------------------------------------------------------------------

def test_full_size_sweep_matrix_int8():
    spec = wl.sweep_spec(0.42)
    w, sc = wl.matrix_inputs(4, 0, 2, spec)
    x = wl.activation_inputs(4, "int8", 1, spec.k)
    rows = _sampled(spec.n, 96, 1)
    ref_raw = O.dense_gemv_raw(w[rows], x).astype(np.int32)
    ref = O.dense_gemv(w[rows], sc.reshape(spec.n, -1)[rows].reshape(-1), 128, x)
    bound = group_bound(w[rows], sc.reshape(spec.n, -1)[rows].reshape(-1), 128, x)
    for fmt in FMTS:
        y, _ = run(fmt, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW)
        assert np.array_equal(y[:, rows], ref_raw)
        y, _ = run(fmt, w, sc, 128, x, "int8")
        check_grouped(y[:, rows], ref, bound)


@pytest.mark.parametrize("midx", [0, 1, 4, 6])
def test_full_size_bitnet_layer_bf16_and_int8(midx):
    wk = wl.WORKLOADS["bitnet2b_layers"]
    spec = wk.matrices[midx]
    w, sc = wl.matrix_inputs(wk.cid, 0, midx, spec)
    xb = wl.activation_inputs(wk.cid, "bf16", 1, spec.k)
    q, a = O.quantize_activations(xb)
    rows = _sampled(spec.n, 64, midx)
    ref_b = O.dense_gemv(w[rows], sc, 0, xb, x_is_bf16_bits=True)
    bound_b = bf16_bound(w[rows], sc, 0, xb)
    ref_q = O.dense_gemv(w[rows], sc, 0, q, a)
    bound_q = group_bound(w[rows], sc, 0, q, a)
    for fmt in FMTS:
        y, _ = run(fmt, w, sc, 0, xb, "bf16")
        check_bf16(y[:, rows], ref_b, bound_b)
        y, _ = run(fmt, w, sc, 0, q, "int8", xscale=a)
        check_grouped(y[:, rows], ref_q, bound_q)


def test_full_size_qwen3_32b_down_nonuniform_rows_int8():
    wk = wl.WORKLOADS["qwen3_32b_layers"]
    spec = wk.matrices[6]       # down: 5120 x 25600, per-row z ~ U[0.30, 0.60]
    w, sc = wl.matrix_inputs(wk.cid, 0, 6, spec)
    x = wl.activation_inputs(wk.cid, "int8", 1, spec.k)
    rows = _sampled(spec.n, 48, 3)
    ref_raw = O.dense_gemv_raw(w[rows], x).astype(np.int32)
    for fmt in FMTS:
        y, _ = run(fmt, w, sc, 128, x, "int8", y_mode=N.Y_I32_RAW)
        assert np.array_equal(y[:, rows], ref_raw)


# ---------------------------------------------------------------------------
# Device activation quantiser (int8 per group of 128), bit-exact vs the oracle
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("m,k", [(1, 128), (1, 2560), (3, 6912), (2, 25600)])
def test_quantize_activations_bit_exact(m, k):
    xb = wl.act_bf16(m, k, wl.rng_for(110, m, k))
    xb[0, :128] = 0                       # an all-zero group -> a = 1
    xb[-1, -5] = 0x4300                   # 128.0: a large outlier
    say("quantize", m, k)
    xd = to_dev_x(xb, "bf16")
    q = torch.empty((m, k), dtype=torch.int8, device="cuda")
    a = torch.empty((m, k // 128), dtype=torch.float32, device="cuda")
    api.quantize_activations(xd, q, a)
    torch.cuda.synchronize()
    qr, ar = O.quantize_activations(xb)
    assert np.array_equal(a.cpu().numpy().view(np.uint32), ar.view(np.uint32))
    assert np.array_equal(q.cpu().numpy(), qr)


# ---------------------------------------------------------------------------
# Batched launch: a list of GEMVs of one tile as one persistent kernel
# ---------------------------------------------------------------------------

def _batch_case(fmt, kind, group, with_xscale=False):
    # Matrices of one K (same tile): different row counts, densities and seeds.
    k = 2560
    specs = [(64, 0.42), (7, 0.0), (640, 0.5), (33, 1.0), (301, 0.467)]
    mats, blobs, xs, ys, scs, refs, bounds, layouts, xss = [], [], [], [], [], [], [], [], []
    for i, (n, z) in enumerate(specs):
        w, sc = inputs(n, k, z, group, 200 + i)
        if kind == "int8":
            x = wl.act_int8(1, k, wl.rng_for(201, i))
            xs_np = None
            if with_xscale:
                xb = wl.act_bf16(1, k, wl.rng_for(202, i))
                x, xs_np = O.quantize_activations(xb)
            ref = O.dense_gemv(w, sc, group, x, xs_np)
            bound = group_bound(w, sc, group, x, xs_np)
        else:
            x = wl.act_bf16(1, k, wl.rng_for(203, i))
            xs_np = None
            ref = O.dense_gemv(w, sc, group, x, x_is_bf16_bits=True)
            bound = bf16_bound(w, sc, group, x)
        L, blob = api.plan_and_pack(fmt, w, sc, group)
        layouts.append(L)
        blobs.append(torch.from_numpy(blob).cuda())
        xs.append(to_dev_x(x, kind).reshape(-1))
        xss.append(None if xs_np is None else torch.from_numpy(np.ascontiguousarray(xs_np, np.float32)).cuda())
        ys.append(torch.full((w.shape[0],), -7.0, dtype=torch.float32, device="cuda"))
        refs.append(ref)
        bounds.append(bound)
    say("batch", FMT_NAME[fmt], kind, f"group={group}", "xscale" if with_xscale else "")
    b = api.Batch(layouts, blobs, xs, ys, xss if with_xscale else None)
    b.run()
    torch.cuda.synchronize()
    for y, ref, bound, kind_ in zip(ys, refs, bounds, [kind] * len(ys)):
        got = y.cpu().numpy()[None]
        if kind == "bf16":
            check_bf16(got, ref, bound)
        elif group == 0 and not with_xscale:
            assert np.array_equal(got, ref)
        else:
            check_grouped(got, ref, bound)
    # a second run gives identical bits
    first = [y.cpu().numpy().copy() for y in ys]
    b.run()
    torch.cuda.synchronize()
    for y, f in zip(ys, first):
        assert np.array_equal(y.cpu().numpy().view(np.uint32), f.view(np.uint32))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("kind,group,xscale", [("int8", 128, False), ("int8", 0, False), ("int8", 0, True),
                                               ("bf16", 0, False), ("bf16", 128, False)])
def test_batch_matches_oracle(fmt, kind, group, xscale):
    _batch_case(fmt, kind, group, xscale)


def test_batch_rejects_mixed_tiles_and_formats():
    w1, s1 = inputs(8, 2560, 0.4, 128, 300)
    w2, s2 = inputs(8, 6912, 0.4, 128, 301)
    L1, b1 = api.plan_and_pack(N.FMT_BITCOS, w1, s1, 128)
    L2, b2 = api.plan_and_pack(N.FMT_BITCOS, w2, s2, 128)
    L3, b3 = api.plan_and_pack(N.FMT_TRIT5, w1, s1, 128)
    dev = lambda a: torch.from_numpy(a).cuda()  # noqa: E731
    x1 = torch.zeros(2560, dtype=torch.int8, device="cuda")
    x2 = torch.zeros(6912, dtype=torch.int8, device="cuda")
    y1 = torch.zeros(8, dtype=torch.float32, device="cuda")
    y2 = torch.zeros(8, dtype=torch.float32, device="cuda")
    with pytest.raises(N.BitcosError) as e:
        api.Batch([L1, L2], [dev(b1), dev(b2)], [x1, x2], [y1, y2])
    assert e.value.status == N.E_UNSUPPORTED
    with pytest.raises(N.BitcosError) as e:
        api.Batch([L1, L3], [dev(b1), dev(b3)], [x1, x1], [y1, y2])
    assert e.value.status == N.E_UNSUPPORTED
