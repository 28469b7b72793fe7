"""Pins for the CPU oracle: values the paper prints, closed forms, brute force, library routines.

Each test names the passage it checks.  A plausible slip in the oracle (a
wrong bit order, a dropped sign, an off-by-one rank, a transposed operand, a
missing scale term) fails at least one of them.
"""

import csv
import ctypes
import os
import shutil
import subprocess
import tempfile
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_csv(name):
    with open(os.path.join(GOLDEN, name)) as f:
        rows = [r for r in f if not r.startswith("#")]
    return list(csv.DictReader(rows))


# ---------------------------------------------------------------------------
# pdep (Sec. II-B, pdep figure)
# ---------------------------------------------------------------------------

def test_pdep_paper_example():
    # Fig. 4: mask 1,0,1,1,0,0,1,0 and a = 1,0,1,1 (bit 0 leftmost) give
    # dst = 1,0,0,1,0,0,1,0.
    mask = sum(b << i for i, b in enumerate([1, 0, 1, 1, 0, 0, 1, 0]))
    a = sum(b << i for i, b in enumerate([1, 0, 1, 1]))
    dst = sum(b << i for i, b in enumerate([1, 0, 0, 1, 0, 0, 1, 0]))
    assert (mask, a, dst) == (0x4D, 0xD, 0x49)
    assert O.pdep32(a, mask) == dst


@pytest.fixture(scope="module")
def host_pdep():
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    with open("/proc/cpuinfo") as f:
        if " bmi2" not in f.read():
            pytest.skip("host CPU lacks BMI2")
    d = tempfile.mkdtemp()
    so = os.path.join(d, "pdep.so")
    src = os.path.join(os.path.dirname(__file__), "helpers", "pdep_bmi2.c")
    subprocess.check_call(["gcc", "-O2", "-mbmi2", "-shared", "-fPIC", src, "-o", so])
    lib = ctypes.CDLL(so)
    lib.host_pdep_u32.restype = ctypes.c_uint32
    lib.host_pdep_u32.argtypes = [ctypes.c_uint32, ctypes.c_uint32]
    return lib.host_pdep_u32


def test_pdep_matches_bmi2(host_pdep):
    rng = np.random.default_rng(7)
    vals = rng.integers(0, 2**32, size=(2000, 2), dtype=np.uint64)
    for a, m in vals:
        assert O.pdep32(int(a), int(m)) == host_pdep(int(a), int(m))
    for m in (0, 0xFFFFFFFF, 0x80000001, 0x55555555):
        for a in (0, 0xFFFFFFFF, 0x12345678):
            assert O.pdep32(a, m) == host_pdep(a, m)


# ---------------------------------------------------------------------------
# Bit order, polarity and Eq. (2): the worked column of Sec. II-C
# ---------------------------------------------------------------------------

def test_worked_column_0xDF():
    col = [+1, +1, +1, +1, -1, 0, -1, +1]
    w = np.zeros((1, 32), dtype=np.int8)
    w[0, :8] = col
    p = O.bitcos_encode(w, np.array([0x3C00], np.uint16), group=0, unit_rows=1)
    bitmap = p.sections[0].view("<u4")
    assert bitmap[0] == 0xDF                       # Eq. (3): p = (1,1,1,1,1,0,1,1)
    assert p.nnz == 7
    stored = [(int(p.sections[1][0]) >> j) & 1 for j in range(7)]
    assert stored == [0, 0, 0, 0, 1, 1, 0]         # only popcount(p) = 7 sign bits
    n = O.pdep32(int(p.sections[1][0]), 0xDF)
    assert [(n >> i) & 1 for i in range(8)] == [0, 0, 0, 0, 1, 0, 1, 0]   # Eq. (3): n
    as_bytes = [O.ternary_from_pn((0xDF >> i) & 1, (n >> i) & 1) & 0xFF for i in range(8)]
    assert as_bytes == [0x01, 0x01, 0x01, 0x01, 0xFF, 0x00, 0xFF, 0x01]
    wd, _ = O.bitcos_decode(p)
    assert wd[0, :8].tolist() == col
    assert O.bitcos_decode_pdep(p)[0, :8].tolist() == col
    assert O.bitcos_decode_lut(p)[0, :8].tolist() == col


# ---------------------------------------------------------------------------
# The (m, s) table, Sec. II-D Eq. (4) and the three-lookup figure
# ---------------------------------------------------------------------------

def test_lut_paper_keys():
    codes, adv = O.lut_entry(0xB6)     # m = 1011b (rows 0, 1, 3), s = 0110b
    assert codes == (+1, -1, 0, -1) and adv == 3
    codes, adv = O.lut_entry(0x66)     # second lookup of the figure: m = 0110b, s = 0110b
    assert codes == (0, +1, -1, 0) and adv == 2


def test_lut_equals_4bit_pdep_composed_with_sign_map():
    for key in range(256):
        m, s = key >> 4, key & 0xF
        n = O.pdep32(s, m)
        expect = tuple(O.ternary_from_pn((m >> i) & 1, (n >> i) & 1) for i in range(4))
        codes, adv = O.lut_entry(key)
        assert codes == expect, hex(key)
        assert adv == bin(m).count("1")


def test_lut_window_overlap_three_groups():
    # Three consecutive groups on one column: cursor advances 3, 2, 3 (figure text);
    # the windows overlap although the consumed bits are disjoint.
    # Keys 0xB6 then 0x66 fix the stream s0..s6 = 0,1,1,0,1,1,0; the third
    # group's nibble is not given, any with three present rows will do.
    m = [0b1011, 0b0110, 0b1101]
    signs = [0, 1, 1, 0, 1, 1, 0, 0]     # 3 + 2 + 3 = 8 compact sign bits
    w = np.zeros((1, 32), np.int8)
    pos = 0
    for g, mg in enumerate(m):
        for i in range(4):
            if (mg >> i) & 1:
                w[0, 4 * g + i] = -1 if signs[pos] else 1
                pos += 1
    p = O.bitcos_encode(w, np.array([0x3C00], np.uint16), group=0)
    stream = int(p.sections[1][0])
    assert (m[0] << 4) | (stream & 0xF) == 0xB6
    assert (m[1] << 4) | ((stream >> 3) & 0xF) == 0x66     # cursor advanced by 3
    assert O.lut_entry(0xB6)[1] + O.lut_entry(0x66)[1] == 5
    assert O.bitcos_decode_lut(p).tolist() == w.tolist()


# ---------------------------------------------------------------------------
# Storage cost, Eq. (1), Sec. I, Table I
# ---------------------------------------------------------------------------

def test_layout_figure_8x8_example():
    # Fig. 2: 30 of 64 weights zero -> 64 presence + 34 sign bits = 1.531 bpw.
    w = wl.ternary_exact(2, 32, 30, wl.rng_for(11))
    p = O.bitcos_encode(w, np.array([0x3C00], np.uint16), group=0)
    assert p.nnz == 34
    sym_bits = p.n * p.k + p.nnz
    assert sym_bits == 98 and round(sym_bits / 64, 3) == 1.531
    assert O.bpw_symbols_bitcos(30 / 64) == pytest.approx(98 / 64)


def test_five_trit_and_two_bit_rates():
    assert O.bpw_trit5() == 1.625                      # ceil(128/5) = 26 bytes / 128
    assert O.bpw_trit5() + O.scale_bits_per_weight(128) == 1.75
    assert O.bpw_bit2() + O.scale_bits_per_weight(128) == 2.125
    # Crossover (Sec. II-A): B(z) = 1.625 exactly at z = 0.375.
    assert O.bpw_symbols_bitcos(0.375) == O.bpw_trit5()
    assert O.bpw_symbols_bitcos(0.376) < O.bpw_trit5() < O.bpw_symbols_bitcos(0.374)


@pytest.mark.parametrize("z", [0.0, 0.3, 0.42, 0.5, 0.95, 1.0])
def test_payload_bpw_is_exactly_two_minus_z_plus_scales(z):
    n, k = 24, 512
    w = wl.ternary(n, k, z, wl.rng_for(3, int(z * 1000)))
    sc = wl.fp16_uniform((n * k // 128,), 0.01, 0.1, wl.rng_for(4))
    p = O.bitcos_encode(w, sc, group=128, unit_rows=4)
    zm = Fraction(int(np.count_nonzero(w == 0)), n * k)
    assert Fraction(O.payload_bits(p), n * k) == 2 - zm + Fraction(1, 8)
    # bitmap bytes, sign bytes and scale bytes individually
    assert len(p.sections[0]) * 8 == n * k
    assert len(p.sections[1]) == (p.nnz + 31) // 32 * 4 + O.bitcos_oracle.SIGN_PAD_BYTES
    assert len(p.sections[3]) == 2 * n * (k // 128)


def test_payload_bits_per_tensor_scale():
    # One fp16 scale for the whole tensor (Table I's BitNet row prints no +scale).
    n, k = 8, 256
    w = wl.ternary(n, k, 0.42, wl.rng_for(31))
    p = O.bitcos_encode(w, np.array([0x2E66], np.uint16), group=0)
    assert O.payload_bits(p) == n * k + int(np.count_nonzero(w)) + 16
    assert O.payload_bits(O.trit5_encode(w, np.array([0x2E66], np.uint16), group=0)) == n * 2 * 26 * 8 + 16
    assert O.payload_bits(O.bit2_encode(w, np.array([0x2E66], np.uint16), group=0)) == 2 * n * k + 16


def test_crossover_exact_bits_at_z_0375():
    n, k = 16, 1024
    w = wl.ternary_exact(n, k, int(0.375 * n * k), wl.rng_for(5))
    sc = wl.fp16_uniform((n * k // 128,), 0.01, 0.1, wl.rng_for(6))
    pb = O.bitcos_encode(w, sc, group=128)
    pt = O.trit5_encode(w, sc, group=128)
    assert O.payload_bits(pb) == O.payload_bits(pt)
    assert len(pt.sections[0]) - O.bitcos_oracle.TRIT5_PAD_BYTES == n * (k // 128) * 26


def test_table1_symbols_and_reductions():
    rows = _read_csv("table1_bitwidths.csv")
    assert len(rows) == 29
    beats_trit5 = 0
    for r in rows:
        z = float(r["zero_pct"]) / 100
        # z is printed to 0.01 % and the rate to 0.001: agree within both roundings.
        assert O.bpw_symbols_bitcos(z) == pytest.approx(float(r["symbols"]), abs=5e-4 + 5e-5), r["model"]
        if r["plus_scale"] == "---":
            # One scale per tensor: compare symbol rates directly.
            bits = O.bpw_symbols_bitcos(z)
            assert round(O.bpw_bit2() / bits, 2) == float(r["bit2_red"])
            assert round(O.bpw_trit5() / bits, 2) == float(r["trit5_red"])
            beats_trit5 += bits < O.bpw_trit5()
            continue
        plus = float(r["plus_scale"])
        overhead = plus - float(r["symbols"])
        # The same measured scale overhead is added to every format.
        assert float(r["bit2_plus_scale"]) == pytest.approx(O.bpw_bit2() + overhead, abs=2e-3)
        assert float(r["trit5_plus_scale"]) == pytest.approx(O.bpw_trit5() + overhead, abs=2e-3)
        assert float(r["bit2_red"]) == pytest.approx(float(r["bit2_plus_scale"]) / plus, abs=6e-3)
        assert float(r["trit5_red"]) == pytest.approx(float(r["trit5_plus_scale"]) / plus, abs=6e-3)
        if r["family"] in ("Bonsai", "CAT-Q"):
            # Group-128 fp16 scales: exactly 16/128 bits per weight on top of 2 - z.
            assert plus == pytest.approx(round(O.bpw_symbols_bitcos(z) + O.scale_bits_per_weight(128), 3), abs=1.1e-3)
            assert float(r["bit2_plus_scale"]) == 2.125 and float(r["trit5_plus_scale"]) == 1.75
        beats_trit5 += plus < float(r["trit5_plus_scale"])
    assert beats_trit5 == 26      # "26 out of the 29 models"
    assert min(float(r["symbols"]) for r in rows) == 1.485


# ---------------------------------------------------------------------------
# Round trips and decode-path agreement (bit-exact, Sec. IV: decodes the same values)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("z", [0.0, 0.3, 0.375, 0.5, 0.95, 1.0])
@pytest.mark.parametrize("group", [128, 0])
def test_round_trip_all_formats(z, group):
    n, k = 13, 384
    w = wl.ternary(n, k, z, wl.rng_for(8, int(z * 1000), group))
    w[3, :] = 0                       # an all-zero row
    w[5, 128:256] = 1                 # an all-non-zero group
    ns = n * (k // 128) if group else 1
    sc = wl.fp16_uniform((ns,), 0.01, 0.1, wl.rng_for(9))
    for unit_rows in (1, 3, 16):
        p = O.bitcos_encode(w, sc, group=group, unit_rows=unit_rows)
        wd, sd = O.bitcos_decode(p)
        assert np.array_equal(wd, w) and np.array_equal(sd, sc)
    pt = O.trit5_encode(w, sc, group=group)
    wd, sd = O.trit5_decode(pt)
    assert np.array_equal(wd, w) and np.array_equal(sd, sc)
    pb = O.bit2_encode(w, sc, group=group)
    wd, sd = O.bit2_decode(pb)
    assert np.array_equal(wd, w) and np.array_equal(sd, sc)


def test_decode_paths_agree():
    w = wl.ternary(6, 256, 0.45, wl.rng_for(10))
    p = O.bitcos_encode(w, wl.fp16_uniform((12,), 0.01, 0.1, wl.rng_for(1)), group=128, unit_rows=2)
    assert np.array_equal(O.bitcos_decode_pdep(p), w)
    assert np.array_equal(O.bitcos_decode_lut(p), w)


def test_unit_offsets_definition():
    w = wl.ternary(10, 256, 0.4, wl.rng_for(12))
    p = O.bitcos_encode(w, np.array([0x3C00], np.uint16), group=0, unit_rows=3)
    off = p.sections[2].view("<u4")
    per_row = (w != 0).sum(axis=1)
    assert off.tolist() == [0, per_row[:3].sum(), per_row[:6].sum(), per_row[:9].sum(), per_row.sum()]


def test_serialize_alignment():
    w = wl.ternary(7, 256, 0.4, wl.rng_for(13))
    p = O.bitcos_encode(w, wl.fp16_uniform((14,), 0.01, 0.1, wl.rng_for(2)), group=128, unit_rows=2)
    blob, offs = O.serialize(p)
    assert len(blob) % 256 == 0
    assert all(o % 256 == 0 for o, _ in offs)
    assert [ln for _, ln in offs] == [len(s) for s in p.sections]
    back = O.deserialize(p, blob, offs)
    assert all(np.array_equal(a, b) for a, b in zip(back, p.sections))


def test_trit5_hand_worked_bytes():
    w = np.zeros((1, 128), np.int8)
    w[0, :5] = [-1, 0, 1, 1, -1]         # digits 0,1,2,2,0 -> 0 + 3 + 18 + 54 + 0
    w[0, 125:128] = [1, 1, 1]            # digits 2,2,2 + pad digits 1,1
    p = O.trit5_encode(w, np.array([0x3C00], np.uint16), group=0)
    b = p.sections[0]
    assert b[0] == 75
    assert b[25] == 2 + 2 * 3 + 2 * 9 + 1 * 27 + 1 * 81
    assert b[1] == sum(3 ** t for t in range(5))       # all-zero weights -> all digits 1 = 121


def test_bit2_hand_worked_word():
    w = np.zeros((1, 128), np.int8)
    w[0, 0] = -1          # t = 0, b = 0 -> code 0 at bits 0..1
    w[0, 1] = +1          # t = 0, b = 1 -> code 2 at bits 8..9
    w[0, 4] = -1          # t = 1, b = 0 -> code 0 at bits 2..3
    p = O.bit2_encode(w, np.array([0x3C00], np.uint16), group=0)
    words = p.sections[0].view("<u4")
    assert words[0] == 0x55555650
    assert words[1] == 0x55555555


# ---------------------------------------------------------------------------
# Dense GEMV: the plain definition (Sec. II-C), against loops and library routines
# ---------------------------------------------------------------------------

def _loop_gemv(w, s_f64, group, x, a):
    n, k = w.shape
    y = np.zeros(n)
    for r in range(n):
        tot = 0.0
        for g in range(k // 128):
            acc = 0
            for kk in range(128 * g, 128 * (g + 1)):
                acc += int(w[r, kk]) * int(x[kk])
            sc = s_f64[r, g] if group == 128 else s_f64[0, 0]
            tot += sc * a[g] * acc
        y[r] = tot
    return y.astype(np.float32)


def test_dense_gemv_raw_matches_triple_loop_and_matmul():
    w = wl.ternary(5, 256, 0.4, wl.rng_for(14))
    x = wl.act_int8(3, 256, wl.rng_for(15))
    y = O.dense_gemv_raw(w, x)
    for m in range(3):
        for r in range(5):
            assert y[m, r] == sum(int(w[r, kk]) * int(x[m, kk]) for kk in range(256))
    assert np.array_equal(y, np.matmul(x.astype(np.int64), w.astype(np.int64).T))


def test_dense_gemv_group_scales_and_activation_scales():
    n, k = 4, 384
    w = wl.ternary(n, k, 0.45, wl.rng_for(16))
    sc = wl.fp16_uniform((n * 3,), 0.01, 0.1, wl.rng_for(17))
    x = wl.act_int8(1, k, wl.rng_for(18))
    a = np.array([0.5, 2.0, 0.25], np.float32)
    s64 = sc.view(np.float16).astype(np.float64).reshape(n, 3)
    ref = _loop_gemv(w, s64, 128, x[0], a.astype(np.float64))
    got = O.dense_gemv(w, sc, 128, x, a.reshape(1, 3))[0]
    assert np.array_equal(got, ref)
    # Swapping two groups' scales must change the answer (catches a transposed S).
    s_bad = sc.reshape(n, 3)[:, ::-1].reshape(-1).copy()
    assert not np.array_equal(O.dense_gemv(w, s_bad, 128, x, a.reshape(1, 3))[0], ref)


def test_dense_gemv_per_tensor_is_one_rounding_of_the_row_sum():
    w = wl.ternary(6, 256, 0.4, wl.rng_for(19))
    x = wl.act_int8(1, 256, wl.rng_for(20))
    s = np.array([np.float16(0.0371).view(np.uint16)], np.uint16)
    y = O.dense_gemv(w, s, 0, x)[0]
    exact = (x.astype(np.int64) @ w.astype(np.int64).T)[0]
    assert np.array_equal(y, (np.float64(np.float16(0.0371)) * exact).astype(np.float32))


def test_dense_gemv_bf16_exact_widening():
    w = wl.ternary(3, 128, 0.3, wl.rng_for(21))
    xb = wl.act_bf16(1, 128, wl.rng_for(22))
    xf = (xb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)[0]
    s = np.array([0x3C00], np.uint16)       # 1.0
    y = O.dense_gemv(w, s, 0, xb, x_is_bf16_bits=True)[0]
    ref = np.array([sum(float(w[r, kk]) * xf[kk] for kk in range(128)) for r in range(3)], np.float32)
    assert np.allclose(y, ref, rtol=1e-6, atol=1e-6)


# ---------------------------------------------------------------------------
# Activation quantisation (Sec. II-C; rule fixed by this build)
# ---------------------------------------------------------------------------

def test_quantize_activations_rule():
    x = np.zeros((1, 256), np.float32)
    x[0, 0] = 127.0
    x[0, 1] = 2.5          # a = 1 -> half-to-even -> 2
    x[0, 2] = -3.5         # -> -4
    x[0, 3] = 0.49
    bits = wl.f32_to_bf16_bits(x)
    q, a = O.quantize_activations(bits)
    assert a.tolist() == [[1.0, 1.0]]          # second group all zero -> a = 1
    assert q[0, :4].tolist() == [127, 2, -4, 0]
    assert not q[0, 128:].any()
    xb = wl.act_bf16(2, 512, wl.rng_for(23))
    q, a = O.quantize_activations(xb)
    xf = O.bf16_bits_to_f64(xb).reshape(2, 4, 128)
    deq = q.reshape(2, 4, 128) * a[:, :, None].astype(np.float64)
    assert np.all(np.abs(deq - xf) <= a[:, :, None] * 0.5 + 1e-6)
    assert np.abs(q).max() == 127


# ---------------------------------------------------------------------------
# Two-term roofline, Sec. III-B1 Eqs. (5)-(6) and Table II
# ---------------------------------------------------------------------------

def test_roofline_bytes_and_table2():
    assert O.roofline_bytes_per_32(0.40) == pytest.approx(6.9)
    assert O.roofline_bytes_per_32(0.95) == pytest.approx(4.7)
    assert round(O.roofline_bytes_per_32(0.95) / 4.60, 2) == 1.02       # EMR at z = 0.95
    for r in _read_csv("table2_roofline.csv"):
        t, e, bound = O.roofline_cpu(0.40, float(r["beta"]), float(r["gamma"]))
        assert 6.9 / float(r["gamma"]) == pytest.approx(float(r["b_over_gamma"]), rel=5e-3)
        assert bound == r["bound"]
        assert e == pytest.approx(min(float(r["beta"]), float(r["b_over_gamma"])), rel=5e-3)
        # Eq. (6): the effective bandwidth is the iteration's bytes over its
        # time, and neither term of Eq. (5) can be beaten: T >= gamma and
        # T >= B / beta, with equality in the term the row is bound by.
        assert t * e == pytest.approx(6.9, rel=1e-12)
        assert t >= float(r["gamma"]) - 1e-12 and t >= 6.9 / float(r["beta"]) - 1e-12
        assert t == pytest.approx(float(r["gamma"]) if bound == "instructions" else 6.9 / float(r["beta"]))


# ---------------------------------------------------------------------------
# Validation
# ---------------------------------------------------------------------------

def test_encoder_rejects_bad_input():
    w = np.zeros((2, 128), np.int8)
    one = np.array([0x3C00, 0x3C00], np.uint16)
    with pytest.raises(ValueError):
        O.bitcos_encode(np.full((2, 128), 2, np.int8), one, 128)
    with pytest.raises(ValueError):
        O.bitcos_encode(w, np.array([0xBC00, 0x3C00], np.uint16), 128)    # negative scale
    with pytest.raises(ValueError):
        O.bitcos_encode(w, np.array([0x7C00, 0x3C00], np.uint16), 128)    # inf
    with pytest.raises(ValueError):
        O.bitcos_encode(np.zeros((2, 100), np.int8), one, 128)
    with pytest.raises(ValueError):
        O.trit5_encode(np.zeros((2, 96), np.int8), np.array([0x3C00], np.uint16), 0)
