"""GPU: the device-side BITCOS packer against the host packer and the oracle.

The host packer writes exactly the oracle's bytes (test_host_lib.py); the
device packer must produce the same layout and the same blob bytes for every
shape, density, scale mode and unit size, and reject what the host packer
rejects.  The packed blob also has to round-trip through the GEMV.
"""

import sys

import numpy as np
import pytest

import oracle as O
import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
api = pytest.importorskip("paper_2609_16338_amd.api")
from paper_2609_16338_amd import _native as N  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    N.lib()


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


LAYOUT_FIELDS = ("version", "format", "n", "k", "group", "unit_rows", "nnz", "total_bytes", "payload_bits")


def device_pack(w, sc, group, unit_rows):
    wd = torch.from_numpy(np.ascontiguousarray(w, dtype=np.int8)).cuda()
    sd = torch.from_numpy(np.ascontiguousarray(sc, dtype=np.uint16).view(np.int16)).cuda()
    return api.bitcos_pack_device(wd, sd, group, unit_rows)


@pytest.mark.parametrize("n,k,z,group,unit", [
    (256, 1024, 0.50, 128, 0),        # the smallest instance
    (37, 256, 0.42, 128, 0),          # ragged rows
    (5, 96, 0.30, 0, 0),              # per-tensor scale, K % 128 != 0
    (64, 2048, 0.0, 128, 1),          # no zeros, one offset per row
    (64, 2048, 1.0, 128, 4),          # all zeros
    (33, 4096 + 128, 0.467, 128, 7),  # ragged words per wave, odd unit
    (1000, 2560, 0.42, 0, 1000),      # one unit for the whole matrix
    (3, 32 * 64 * 3 + 32, 0.6, 0, 2), # several 64-word passes per row
])
def test_device_pack_matches_host(n, k, z, group, unit):
    rng = wl.rng_for(71, n, k, int(z * 1000))
    w = wl.ternary(n, k, z, rng)
    ns = n * (k // 128) if group == 128 else 1
    sc = wl.fp16_uniform((ns,), 0.01, 0.1, wl.rng_for(72, n, k))
    say("pack_device", (n, k), f"z={z}", f"group={group}", f"unit={unit}")
    Lh, blob_h = api.plan_and_pack(N.FMT_BITCOS, w, sc, group, unit)
    Ld, blob_d = device_pack(w, sc, group, unit)
    for f in LAYOUT_FIELDS:
        assert getattr(Ld, f) == getattr(Lh, f), f
    assert list(Ld.sec_off) == list(Lh.sec_off) and list(Ld.sec_bytes) == list(Lh.sec_bytes)
    got = blob_d.cpu().numpy()
    assert got.shape == blob_h.shape
    bad = np.flatnonzero(got != blob_h)
    assert bad.size == 0, f"{bad.size} bytes differ, first at {bad[:8]}"
    # and the oracle's own serialised blob, byte for byte
    ob, _ = O.serialize(O.bitcos_encode(w, sc, group, Lh.unit_rows))
    assert np.array_equal(got, np.frombuffer(ob, dtype=np.uint8))


def test_device_pack_full_size_and_gemv():
    spec = wl.sweep_spec(0.42)
    w, sc = wl.matrix_inputs(4, 0, 2, spec)
    say("pack_device full size", (spec.n, spec.k))
    Lh, blob_h = api.plan_and_pack(N.FMT_BITCOS, w, sc, spec.group)
    Ld, blob_d = device_pack(w, sc, spec.group, 0)
    assert Ld.total_bytes == Lh.total_bytes and Ld.nnz == Lh.nnz
    assert np.array_equal(blob_d.cpu().numpy(), blob_h)
    # the device blob drives the GEMV: raw int32 sums on sampled rows
    x = wl.activation_inputs(4, "int8", 1, spec.k)
    xd = torch.from_numpy(x).cuda()
    y = torch.empty((1, spec.n), dtype=torch.int32, device="cuda")
    api.gemv(Ld, blob_d, xd, y, y_mode=N.Y_I32_RAW)
    torch.cuda.synchronize()
    rows = np.arange(0, spec.n, 97)
    ref = O.dense_gemv_raw(w[rows], x)
    assert np.array_equal(y.cpu().numpy()[:, rows], ref)


def test_device_pack_rejects_bad_values():
    w = wl.ternary(8, 256, 0.4, wl.rng_for(73))
    sc = wl.fp16_uniform((16,), 0.01, 0.1, wl.rng_for(74))
    bad_w = w.copy()
    bad_w[3, 17] = 2
    say("pack_device rejects weight 2")
    with pytest.raises(N.BitcosError) as e:
        device_pack(bad_w, sc, 128, 0)
    assert e.value.status == N.E_VALUE
    bad_s = sc.copy()
    bad_s[5] = 0xBC00  # -1.0
    say("pack_device rejects a negative scale")
    with pytest.raises(N.BitcosError) as e:
        device_pack(w, bad_s, 128, 0)
    assert e.value.status == N.E_VALUE
    bad_s[5] = 0x7C00  # +inf
    with pytest.raises(N.BitcosError) as e:
        device_pack(w, bad_s, 128, 0)
    assert e.value.status == N.E_VALUE


def test_device_pack_detects_changed_weights():
    """W changed between plan and pack: E_VALUE, and nothing outside the blob is touched."""
    lib = N.lib()
    import ctypes
    n, k = 16, 512
    w = wl.ternary(n, k, 0.5, wl.rng_for(75))
    sc = wl.fp16_uniform((n * k // 128,), 0.01, 0.1, wl.rng_for(76))
    wd = torch.from_numpy(w).cuda()
    sd = torch.from_numpy(sc.view(np.int16)).cuda()
    ws_bytes = lib.bitcos_plan_device_workspace(n)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    L = N.Layout()
    N.check(lib.bitcos_plan_device(ctypes.c_void_p(wd.data_ptr()), n, k, 128, 0, ctypes.c_void_p(ws.data_ptr()),
                                   ws_bytes, ctypes.byref(L), None), "plan")
    w2 = w.copy()
    w2[w2 == 0] = 1  # more non-zeros than planned
    wd2 = torch.from_numpy(w2).cuda()
    guard = 4096
    buf = torch.full((L.total_bytes + 2 * guard,), 0x5A, dtype=torch.uint8, device="cuda")
    say("pack_device with changed weights")
    st = lib.bitcos_pack_device(ctypes.c_void_p(wd2.data_ptr()), ctypes.c_void_p(sd.data_ptr()), ctypes.byref(L),
                                ctypes.c_void_p(ws.data_ptr()), ws_bytes,
                                ctypes.c_void_p(buf.data_ptr() + guard), L.total_bytes, None)
    assert st == N.E_VALUE
    b = buf.cpu().numpy()
    assert (b[:guard] == 0x5A).all() and (b[guard + L.total_bytes:] == 0x5A).all()


def test_device_pack_argument_errors():
    lib = N.lib()
    import ctypes
    L = N.Layout()
    assert lib.bitcos_plan_device_workspace(0) == 0
    assert lib.bitcos_plan_device(None, 4, 128, 128, 0, None, 0, ctypes.byref(L), None) == N.E_ARG
    wd = torch.zeros((4, 100), dtype=torch.int8, device="cuda")
    ws = torch.empty(256, dtype=torch.uint8, device="cuda")
    # K not a multiple of 128 with group scales
    assert lib.bitcos_plan_device(ctypes.c_void_p(wd.data_ptr()), 4, 100, 128, 0, ctypes.c_void_p(ws.data_ptr()),
                                  256, ctypes.byref(L), None) == N.E_ARG
    # workspace too small
    wd = torch.zeros((64, 128), dtype=torch.int8, device="cuda")
    assert lib.bitcos_plan_device(ctypes.c_void_p(wd.data_ptr()), 64, 128, 128, 0, ctypes.c_void_p(ws.data_ptr()),
                                  16, ctypes.byref(L), None) == N.E_SPACE
