"""GPU parity on seeded random shapes, through the C ABI.

Sixty cases drawn from one seed over everything the launcher routes on: row
count (1 to 600), K (multiples of 32, or of 128 where scale groups or several
activation rows need it, up to rows longer than the batch-1 kernels hold),
zero density (including 0 and 1), per-tensor or group-128 scales, int8 or
bf16 activations, 1 to 16 activation rows, activation scales and raw int32
sums.  Every case is checked against the oracle in full, to the same bars as
the other parity tests: raw sums and per-tensor int8 bit-exact; group- or
activation-scaled int8 within 1e-5 of sum_g |S a A|; bf16 within 1e-3 of
sum |S W x| per element and in norm.
"""

import numpy as np
import pytest

import oracle as O
import workloads as wl
from parity_checks import bf16_bound, check_bf16, check_grouped, group_bound, inputs, run

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
api = pytest.importorskip("paper_2609_16338_amd.api")
from paper_2609_16338_amd import _native as N  # noqa: E402

CASES = 60
MAX_WEIGHTS = 3_000_000  # per case, so that the oracle stays fast


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    N.lib()


def draw(i):
    rng = wl.rng_for(900, i)
    kind = "int8" if rng.random() < 0.5 else "bf16"
    m = 1 if rng.random() < 0.75 else int(rng.choice([2, 3, 4, 7, 16]))
    group = 128 if rng.random() < 0.6 else 0
    long_row = rng.random() < 0.15
    step = 128 if (group or m > 1 or long_row) else 32
    kmax = (16384 if kind == "bf16" else 32768) if m == 1 and not long_row else 25600
    kmin = (16512 if kind == "bf16" else 32896) if (m == 1 and long_row) else step
    if kmin > kmax:
        kmax = kmin + 128 * 8
    k = int(rng.integers(kmin // step, kmax // step + 1)) * step
    n = int(rng.integers(1, max(2, min(600, MAX_WEIGHTS // k)) + 1))
    zc = rng.random()
    z = 0.0 if zc < 0.08 else 1.0 if zc < 0.14 else float(rng.uniform(0.2, 0.8))
    xscale = kind == "int8" and k % 128 == 0 and rng.random() < 0.4
    raw = kind == "int8" and not xscale and rng.random() < 0.4
    return dict(kind=kind, m=m, group=group, k=k, n=n, z=z, xscale=xscale, raw=raw)


def test_draws_cover_the_routes():
    cs = [draw(i) for i in range(CASES)]
    assert {c["kind"] for c in cs} == {"int8", "bf16"}
    assert any(c["m"] > 1 for c in cs) and any(c["m"] == 1 for c in cs)
    assert any(c["k"] > 16384 and c["kind"] == "bf16" and c["m"] == 1 for c in cs)
    assert any(c["z"] == 0.0 for c in cs) and any(c["z"] == 1.0 for c in cs)
    assert any(c["xscale"] for c in cs) and any(c["raw"] for c in cs)
    assert any(c["k"] % 128 for c in cs)


@pytest.mark.parametrize("i", range(CASES))
def test_random_shape(i):
    c = draw(i)
    w, sc = inputs(c["n"], c["k"], c["z"], c["group"], 910 + i)
    xr = wl.rng_for(920, i)
    a = None
    if c["kind"] == "bf16":
        x = wl.act_bf16(c["m"], c["k"], xr)
    elif c["xscale"]:
        x, a = O.quantize_activations(wl.act_bf16(c["m"], c["k"], xr))
    else:
        x = wl.act_int8(c["m"], c["k"], xr)
    if c["raw"]:
        y, _ = run(N.FMT_BITCOS, w, sc, c["group"], x, "int8", y_mode=N.Y_I32_RAW)
        assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32)), c
        return
    y, _ = run(N.FMT_BITCOS, w, sc, c["group"], x, c["kind"], xscale=a)
    if c["kind"] == "bf16":
        ref = O.dense_gemv(w, sc, c["group"], x, x_is_bf16_bits=True)
        check_bf16(y, ref, bf16_bound(w, sc, c["group"], x))
    elif c["group"] == 0 and a is None:
        assert np.array_equal(y, O.dense_gemv(w, sc, 0, x)), c
    else:
        ref = O.dense_gemv(w, sc, c["group"], x, xscale=a)
        check_grouped(y, ref, group_bound(w, sc, c["group"], x, a))


BASELINE_CASES = 30


def draw_baseline(i):
    rng = wl.rng_for(930, i)
    fmt = N.FMT_TRIT5 if rng.random() < 0.5 else N.FMT_BIT2
    kind = "int8" if rng.random() < 0.5 else "bf16"
    m = 1 if rng.random() < 0.8 else int(rng.choice([2, 5]))
    group = 128 if rng.random() < 0.6 else 0
    kmax = 16384 if kind == "bf16" else 32768
    k = int(rng.integers(1, kmax // 128 + 1)) * 128
    n = int(rng.integers(1, max(2, min(400, MAX_WEIGHTS // k)) + 1))
    zc = rng.random()
    z = 0.0 if zc < 0.1 else 1.0 if zc < 0.2 else float(rng.uniform(0.2, 0.8))
    xscale = kind == "int8" and rng.random() < 0.4
    raw = kind == "int8" and not xscale and rng.random() < 0.4
    return dict(fmt=fmt, kind=kind, m=m, group=group, k=k, n=n, z=z, xscale=xscale, raw=raw)


@pytest.mark.parametrize("i", range(BASELINE_CASES))
def test_random_shape_baselines(i):
    """The five-trit and 2-bit kernels on seeded random shapes, same bars."""
    c = draw_baseline(i)
    w, sc = inputs(c["n"], c["k"], c["z"], c["group"], 940 + i)
    xr = wl.rng_for(950, i)
    a = None
    if c["kind"] == "bf16":
        x = wl.act_bf16(c["m"], c["k"], xr)
    elif c["xscale"]:
        x, a = O.quantize_activations(wl.act_bf16(c["m"], c["k"], xr))
    else:
        x = wl.act_int8(c["m"], c["k"], xr)
    if c["raw"]:
        y, _ = run(c["fmt"], w, sc, c["group"], x, "int8", y_mode=N.Y_I32_RAW)
        assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32)), c
        return
    y, _ = run(c["fmt"], w, sc, c["group"], x, c["kind"], xscale=a)
    if c["kind"] == "bf16":
        ref = O.dense_gemv(w, sc, c["group"], x, x_is_bf16_bits=True)
        check_bf16(y, ref, bf16_bound(w, sc, c["group"], x))
    elif c["group"] == 0 and a is None:
        assert np.array_equal(y, O.dense_gemv(w, sc, 0, x)), c
    else:
        ref = O.dense_gemv(w, sc, c["group"], x, xscale=a)
        check_grouped(y, ref, group_bound(w, sc, c["group"], x, a))
