"""Slow, obviously-correct CPU oracle for the BITCOS hot path.

TEST INFRASTRUCTURE ONLY -- see ``oracle/__init__.py``.  Written from the
paper "Breaking the 1.58-bit Barrier for Ternary LLMs" (Georganas, Heinecke,
Dubey); citations name the paper's section, equation, figure or table.

What the oracle computes
------------------------
* ``pdep32``          -- the parallel bit deposit defined in the pdep figure
                         of Sec. II-B (Fig. 4): bits of the source, taken in
                         order, land on the set bits of the mask.
* ``lut_entry``       -- the 256-entry (m, s) table of Sec. II-D, Eq. (4):
                         c_i = 0 if m_i = 0, else +1/-1 for sign bit
                         s_{r_i} = 0/1, with r_i the rank of row i among the
                         present rows of the nibble.
* ``ternary_from_pn`` -- Sec. II-C, Eq. (2): w = p - 2n.
* ``bitcos_encode`` / ``bitcos_decode`` -- the layout of Sec. II-A: a dense
                         presence bitmap (one bit per weight, set where the
                         weight is non-zero) and a sign vector with one bit per
                         non-zero in the same tensor order (the j-th sign bit
                         belongs to the j-th set bit; a set sign bit means
                         negative, Eq. (4)).  Plus the per-unit sign offsets
                         and the group scales this build stores beside them.
* ``bitcos_decode_pdep`` / ``bitcos_decode_lut`` -- the same decode done the
                         way the unpack sequences do it: per 32-bit presence
                         word a pdep of the next sign bits (Sec. II-B/C), or
                         per presence nibble a table lookup keyed by
                         (m << 4) | s with the cursor advancing by popcount(m)
                         (Sec. II-D, the three-lookup figure, Fig. 9).
* ``trit5_encode`` / ``trit5_decode`` -- five trits per byte, 26 bytes per
                         128-weight block (Sec. I).  The digit order inside a
                         block is this build's choice (the paper gives only
                         the rate): parity of the encoding itself is pinned
                         only by round trip, exact size and a hand-worked
                         byte.
* ``bit2_encode`` / ``bit2_decode`` -- 2 bits per weight (Table I's 2-bit
                         column).  Field order is this build's choice; pinned
                         as for trit5.
* ``dense_gemv``      -- the plain definition the GEMV must reach:
                         y[n] = sum_g S[n,g] * a_g * sum_{k in g} W[n,k] x[k],
                         integer-exact for int8 x, float64 otherwise, rounded
                         once to fp32 (Sec. II-C: int8 activations, int32
                         accumulation, scale applied once per group).
* ``quantize_activations`` -- int8 per group of 128 (Sec. II-C).  The paper
                         does not state the rule; this oracle takes
                         a = max|x| / 127 in fp32 (a = 1 for an all-zero
                         group) and q = clamp(round_half_even(x / a), -127,
                         127) with the division in fp32.
* ``bpw_*``           -- storage accounting: B(z) = 2 - z (Sec. II-A,
                         Eq. (1)), the five-trit 26 B / 128 rate (Sec. I),
                         2-bit, plus 16 bits per scale group (Table I).
* ``roofline_cpu``    -- the two-term model of Sec. III-B1, Eqs. (5)-(6).

Blob serialisation (shared *specification*, implemented independently here
and in the C++ library): every section starts at a 256-byte boundary of the
blob, in the order bitmap, signs, unit offsets, scales (BITCOS) or codes,
scales (five-trit, 2-bit); the blob length is rounded up to 256 bytes.

Parity status: every function above is pinned by the tests in
``tests/test_oracle_pins.py`` against values the paper prints, closed forms,
brute force or library routines -- except the *internal digit/field order* of
the two in-house baseline formats (trit5, bit2), which the paper does not
define: parity unpinned beyond round trip, size and hand-worked bytes.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "ALIGN",
    "FMT_BITCOS",
    "FMT_TRIT5",
    "FMT_BIT2",
    "pdep32",
    "popcount",
    "lut_entry",
    "lut_table",
    "ternary_from_pn",
    "Packed",
    "bitcos_encode",
    "bitcos_decode",
    "bitcos_decode_pdep",
    "bitcos_decode_lut",
    "trit5_encode",
    "trit5_decode",
    "bit2_encode",
    "bit2_decode",
    "serialize",
    "deserialize",
    "dense_gemv",
    "dense_gemv_raw",
    "gemv_from_packed",
    "quantize_activations",
    "bpw_symbols_bitcos",
    "bpw_payload",
    "payload_bits",
    "bpw_trit5",
    "bpw_bit2",
    "scale_bits_per_weight",
    "roofline_cpu",
    "roofline_bytes_per_32",
    "fp16_bits_to_f64",
    "bf16_bits_to_f64",
]

ALIGN = 256
FMT_BITCOS = 1
FMT_TRIT5 = 2
FMT_BIT2 = 3


# ---------------------------------------------------------------------------
# Bit primitives
# ---------------------------------------------------------------------------

def popcount(v: int) -> int:
    """Number of set bits of a non-negative integer."""
    return bin(int(v)).count("1")


def pdep32(a: int, mask: int) -> int:
    """Parallel bit deposit (Sec. II-B, pdep figure, Fig. 4).

    Walk the 32 mask positions from bit 0 up; at every set mask bit, copy the
    next not-yet-used low bit of ``a`` there.  Unselected positions are zero.
    """
    dst = 0
    k = 0
    for m in range(32):
        if (mask >> m) & 1:
            if (a >> k) & 1:
                dst |= 1 << m
            k += 1
    return dst


def ternary_from_pn(p: int, n: int) -> int:
    """Sec. II-C, Eq. (2): a present weight is +1, or -1 when negative."""
    return p - 2 * n


def lut_entry(key: int) -> tuple[tuple[int, int, int, int], int]:
    """Entry of the 256-entry table, Sec. II-D, Eq. (4).

    ``key = (m << 4) | s``: m is the presence nibble (bit i = row i of the
    four-row group), s the next four bits of the compact sign stream.
    Returns the four ternary codes and the cursor advance popcount(m).
    """
    m = (key >> 4) & 0xF
    s = key & 0xF
    codes = []
    for i in range(4):
        if not (m >> i) & 1:
            codes.append(0)
            continue
        r_i = sum((m >> j) & 1 for j in range(i))  # rank among present rows
        codes.append(-1 if (s >> r_i) & 1 else +1)
    return tuple(codes), popcount(m)


def lut_table() -> list[tuple[tuple[int, int, int, int], int]]:
    return [lut_entry(key) for key in range(256)]


# ---------------------------------------------------------------------------
# Numeric helpers for stored bit patterns
# ---------------------------------------------------------------------------

def fp16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


# ---------------------------------------------------------------------------
# Packed container and serialisation
# ---------------------------------------------------------------------------

@dataclass
class Packed:
    fmt: int
    n: int
    k: int
    group: int               # 128, or 0 for one scale per tensor
    unit_rows: int           # BITCOS only: rows per sign-offset entry
    nnz: int
    sections: list = field(default_factory=list)   # list of np.uint8 arrays
    scales: np.ndarray | None = None                # uint16 fp16 bits

    def num_scales(self) -> int:
        return self.n * (self.k // 128) if self.group == 128 else 1


def _round_up(v: int, a: int) -> int:
    return (v + a - 1) // a * a


def serialize(p: Packed) -> tuple[bytes, list[tuple[int, int]]]:
    """Lay the sections out at 256-byte boundaries; return (blob, [(off, len)])."""
    offs = []
    pos = 0
    for sec in p.sections:
        pos = _round_up(pos, ALIGN)
        offs.append((pos, len(sec)))
        pos += len(sec)
    total = _round_up(pos, ALIGN)
    blob = bytearray(total)
    for (o, ln), sec in zip(offs, p.sections):
        blob[o:o + ln] = bytes(sec)
    return bytes(blob), offs


def deserialize(p_meta: Packed, blob: bytes, offs) -> list[np.ndarray]:
    return [np.frombuffer(blob, dtype=np.uint8, count=ln, offset=o).copy() for (o, ln) in offs]


# ---------------------------------------------------------------------------
# Validation shared by the three encoders (plain checks, not arithmetic)
# ---------------------------------------------------------------------------

def _check_inputs(w: np.ndarray, scales: np.ndarray, group: int, need_k_mult: int) -> tuple[int, int]:
    w = np.asarray(w)
    if w.ndim != 2 or w.dtype != np.int8:
        raise ValueError("W must be a 2-D int8 array")
    n, k = w.shape
    if n < 1 or k < 1:
        raise ValueError("empty matrix")
    if group not in (0, 128):
        raise ValueError("group must be 128 or 0 (per tensor)")
    if k % need_k_mult:
        raise ValueError(f"K must be a multiple of {need_k_mult}")
    if np.any((w < -1) | (w > 1)):
        raise ValueError("weights must be in {-1, 0, +1}")
    ns = n * (k // 128) if group == 128 else 1
    sc = np.asarray(scales, dtype=np.uint16).reshape(-1)
    if sc.size != ns:
        raise ValueError(f"expected {ns} scales, got {sc.size}")
    f = fp16_bits_to_f64(sc)
    if not np.all(np.isfinite(f)) or np.any(np.signbit(f) & (f != 0)) or np.any(sc & 0x8000):
        raise ValueError("scales must be finite and non-negative")
    return n, k


def _bits_to_u32_le(bits: np.ndarray) -> np.ndarray:
    """Pack a 0/1 array LSB-first into little-endian uint32 words (zero tail)."""
    bits = np.asarray(bits, dtype=np.uint8)
    nwords = (bits.size + 31) // 32
    padded = np.zeros(nwords * 32, dtype=np.uint8)
    padded[: bits.size] = bits
    return np.packbits(padded, bitorder="little").view("<u4")


def _u32_to_bits(words: np.ndarray, count: int) -> np.ndarray:
    return np.unpackbits(np.asarray(words, dtype="<u4").view(np.uint8), bitorder="little")[:count]


# ---------------------------------------------------------------------------
# BITCOS layout (Sec. II-A)
# ---------------------------------------------------------------------------

SIGN_PAD_BYTES = 16


def bitcos_encode(w: np.ndarray, scales: np.ndarray, group: int = 128, unit_rows: int = 1) -> Packed:
    """Encode W (N x K, int8 in {-1,0,1}) as bitmap + compacted signs.

    Tensor order is row-major (n, k): flat index i = n*K + k.  Bitmap word
    ``w`` bit ``b`` is element 32w + b (least significant bit first, the bit
    order of the 0xDF worked column, Sec. II-C).  The sign stream holds one bit
    per non-zero, in the same order, 1 = negative (Eq. (4)), followed by
    ``SIGN_PAD_BYTES`` zero bytes.  ``off[u]`` counts the non-zeros in rows
    [0, u * unit_rows); the last entry is nnz.
    """
    n, k = _check_inputs(w, scales, group, 128 if group == 128 else 32)
    if unit_rows < 1:
        raise ValueError("unit_rows must be >= 1")
    flat = np.asarray(w, dtype=np.int8).reshape(-1)
    present = (flat != 0).astype(np.uint8)
    negative = (flat[flat != 0] < 0).astype(np.uint8)     # j-th non-zero's sign
    nnz = int(present.sum())

    bitmap = _bits_to_u32_le(present)
    assert bitmap.size == n * k // 32
    signs = _bits_to_u32_le(negative)
    signs_bytes = np.concatenate([signs.view(np.uint8), np.zeros(SIGN_PAD_BYTES, np.uint8)])

    nunits = (n + unit_rows - 1) // unit_rows
    per_row = present.reshape(n, k).sum(axis=1, dtype=np.int64)
    off = np.zeros(nunits + 1, dtype=np.int64)
    for u in range(1, nunits + 1):
        off[u] = off[u - 1] + per_row[(u - 1) * unit_rows: min(u * unit_rows, n)].sum()
    assert off[-1] == nnz
    if nnz >= 2**32:
        raise ValueError("nnz does not fit the 32-bit sign offsets")

    sc = np.asarray(scales, dtype=np.uint16).reshape(-1)
    return Packed(
        fmt=FMT_BITCOS, n=n, k=k, group=group, unit_rows=unit_rows, nnz=nnz,
        sections=[bitmap.view(np.uint8), signs_bytes, off.astype("<u4").view(np.uint8),
                  sc.astype("<u2").view(np.uint8)],
        scales=sc.copy(),
    )


def bitcos_decode(p: Packed) -> tuple[np.ndarray, np.ndarray]:
    """Exact inverse: walk the bitmap and take the next sign bit at each set bit."""
    n, k = p.n, p.k
    present = _u32_to_bits(p.sections[0].view("<u4"), n * k).astype(bool)
    nnz = int(present.sum())
    if nnz != p.nnz:
        raise ValueError("bitmap popcount does not match nnz")
    neg = _u32_to_bits(p.sections[1][: (nnz + 31) // 32 * 4].view("<u4"), nnz)
    flat = np.zeros(n * k, dtype=np.int8)
    flat[present] = (1 - 2 * neg.astype(np.int16)).astype(np.int8)
    _check_offsets(p, present.reshape(n, k))
    return flat.reshape(n, k), p.sections[3].view("<u2").copy()


def _check_offsets(p: Packed, present2d: np.ndarray) -> None:
    off = p.sections[2].view("<u4").astype(np.int64)
    nunits = (p.n + p.unit_rows - 1) // p.unit_rows
    if off.size != nunits + 1:
        raise ValueError("wrong number of unit offsets")
    run = 0
    for u in range(nunits):
        if off[u] != run:
            raise ValueError(f"unit offset {u} is {off[u]}, expected {run}")
        run += int(present2d[u * p.unit_rows: (u + 1) * p.unit_rows].sum())
    if off[nunits] != run:
        raise ValueError("last unit offset is not nnz")


def _sign_window(sign_bits: np.ndarray, cursor: int, width: int) -> int:
    """Integer made of ``width`` sign bits starting at ``cursor`` (LSB first)."""
    seg = sign_bits[cursor: cursor + width]
    v = 0
    for i, b in enumerate(seg):
        v |= int(b) << i
    return v


def bitcos_decode_pdep(p: Packed) -> np.ndarray:
    """Decode word by word as the x86 sequences do (Sec. II-B/C).

    For each 32-bit presence word P: the next 32 compact sign bits at the
    cursor are deposited onto the set bits of P (pdep), giving the per-row
    negative flags n; w = p - 2n (Eq. (2)); the cursor advances by popcount(P).
    Pure-Python loops: small inputs only.
    """
    words = p.sections[0].view("<u4")
    sign_bits = _u32_to_bits(p.sections[1].view(np.uint8)[: len(p.sections[1]) // 4 * 4].view("<u4"),
                             len(p.sections[1]) // 4 * 32)
    out = np.zeros(p.n * p.k, dtype=np.int8)
    cursor = 0
    for wi, P in enumerate(words):
        P = int(P)
        nflags = pdep32(_sign_window(sign_bits, cursor, 32), P)
        for b in range(32):
            out[32 * wi + b] = ternary_from_pn((P >> b) & 1, (nflags >> b) & 1)
        cursor += popcount(P)
    return out.reshape(p.n, p.k)


def bitcos_decode_lut(p: Packed) -> np.ndarray:
    """Decode nibble by nibble with the Eq. (4) table (Sec. II-D, Fig. 9).

    Each four-weight group forms key = (m << 4) | s from its presence nibble m
    and the next four compact sign bits s at the cursor; the entry gives the
    four codes and the cursor advances by popcount(m) only, so successive
    windows overlap.  Pure-Python loops: small inputs only.
    """
    table = lut_table()
    words = p.sections[0].view("<u4")
    nbits = len(p.sections[1]) // 4 * 32
    sign_bits = _u32_to_bits(p.sections[1][: nbits // 8].view("<u4"), nbits)
    out = np.zeros(p.n * p.k, dtype=np.int8)
    cursor = 0
    for wi, P in enumerate(words):
        P = int(P)
        for g in range(8):
            m = (P >> (4 * g)) & 0xF
            s = _sign_window(sign_bits, cursor, 4)
            codes, adv = table[(m << 4) | s]
            out[32 * wi + 4 * g: 32 * wi + 4 * g + 4] = codes
            cursor += adv
    return out.reshape(p.n, p.k)


# ---------------------------------------------------------------------------
# Five-trit baseline (Sec. I: 3^5 = 243 <= 256, 26 bytes per 128 weights)
# ---------------------------------------------------------------------------

TRIT5_BLOCK_BYTES = 26
TRIT5_PAD_BYTES = 16


def trit5_encode(w: np.ndarray, scales: np.ndarray, group: int = 128) -> Packed:
    """Five ternary digits per byte, 26 bytes per 128-weight block along K.

    Blocks are row-major [N][K/128].  Byte j of a block holds weights
    5j .. 5j+4 of the block (only those < 128): digit d_t = w + 1 of weight
    5j + t, byte value sum_t d_t * 3**t.  Missing digits of byte 25 (weights
    128, 129 do not exist) are the digit 1, i.e. weight 0.
    """
    n, k = _check_inputs(w, scales, group, 128)
    wr = np.asarray(w, dtype=np.int8).reshape(n, k // 128, 128)
    out = np.zeros((n, k // 128, TRIT5_BLOCK_BYTES), dtype=np.uint8)
    for j in range(TRIT5_BLOCK_BYTES):
        val = np.zeros((n, k // 128), dtype=np.int32)
        for t in range(5):
            idx = 5 * j + t
            d = (wr[:, :, idx].astype(np.int32) + 1) if idx < 128 else np.ones((n, k // 128), np.int32)
            val += d * 3 ** t
        out[:, :, j] = val.astype(np.uint8)
    codes = np.concatenate([out.reshape(-1), np.zeros(TRIT5_PAD_BYTES, np.uint8)])
    sc = np.asarray(scales, dtype=np.uint16).reshape(-1)
    return Packed(FMT_TRIT5, n, k, group, 0, int(np.count_nonzero(w)),
                  [codes, sc.astype("<u2").view(np.uint8)], sc.copy())


def trit5_decode(p: Packed) -> tuple[np.ndarray, np.ndarray]:
    n, k = p.n, p.k
    nb = n * (k // 128)
    codes = p.sections[0][: nb * TRIT5_BLOCK_BYTES].reshape(n, k // 128, TRIT5_BLOCK_BYTES).astype(np.int32)
    if np.any(codes > 242):
        raise ValueError("five-trit byte above 3**5 - 1")
    w = np.zeros((n, k // 128, 128), dtype=np.int8)
    for j in range(TRIT5_BLOCK_BYTES):
        v = codes[:, :, j].copy()
        for t in range(5):
            d = v % 3
            v //= 3
            idx = 5 * j + t
            if idx < 128:
                w[:, :, idx] = (d - 1).astype(np.int8)
            elif np.any(d != 1):
                raise ValueError("five-trit pad digit is not 1")
    return w.reshape(n, k), p.sections[1].view("<u2").copy()


# ---------------------------------------------------------------------------
# 2-bit baseline (Table I's 2-bit column: 2 bits per weight)
# ---------------------------------------------------------------------------

def bit2_encode(w: np.ndarray, scales: np.ndarray, group: int = 128) -> Packed:
    """Code c = w + 1 in {0, 1, 2}, 16 weights per little-endian u32.

    In the u32 that holds weights k0 .. k0+15 (k0 a multiple of 16), weight
    k0 + 4t + b sits at bits [8b + 2t, 8b + 2t + 1].
    """
    n, k = _check_inputs(w, scales, group, 128)
    c = (np.asarray(w, dtype=np.int8).astype(np.uint32) + 1) & 3
    c = c.reshape(n, k // 16, 4, 4)          # [..., t, b]
    word = np.zeros((n, k // 16), dtype=np.uint32)
    for t in range(4):
        for b in range(4):
            word |= c[:, :, t, b] << np.uint32(8 * b + 2 * t)
    sc = np.asarray(scales, dtype=np.uint16).reshape(-1)
    return Packed(FMT_BIT2, n, k, group, 0, int(np.count_nonzero(w)),
                  [word.astype("<u4").view(np.uint8).reshape(-1), sc.astype("<u2").view(np.uint8)], sc.copy())


def bit2_decode(p: Packed) -> tuple[np.ndarray, np.ndarray]:
    n, k = p.n, p.k
    word = p.sections[0].view("<u4").reshape(n, k // 16)
    w = np.zeros((n, k // 16, 4, 4), dtype=np.int8)
    for t in range(4):
        for b in range(4):
            code = (word >> np.uint32(8 * b + 2 * t)) & 3
            if np.any(code == 3):
                raise ValueError("2-bit code 3 is invalid")
            w[:, :, t, b] = code.astype(np.int8) - 1
    return w.reshape(n, k), p.sections[1].view("<u2").copy()


# ---------------------------------------------------------------------------
# Dense GEMV: the plain definition the packed GEMV must reach
# ---------------------------------------------------------------------------

def _expand_scales(scales_bits: np.ndarray, n: int, k: int, group: int) -> np.ndarray:
    s = fp16_bits_to_f64(np.asarray(scales_bits).reshape(-1))
    if group == 128:
        return s.reshape(n, k // 128)
    return np.full((n, max(k // 128, 1)), s[0])


def dense_gemv_raw(w: np.ndarray, x: np.ndarray) -> np.ndarray:
    """y[m, n] = sum_k W[n, k] * x[m, k] exactly (int64); x is M x K integers."""
    w64 = np.asarray(w, dtype=np.int64)
    x64 = np.atleast_2d(np.asarray(x, dtype=np.int64))
    return x64 @ w64.T


def dense_gemv(w: np.ndarray, scales_bits: np.ndarray, group: int, x: np.ndarray,
               xscale: np.ndarray | None = None, x_is_bf16_bits: bool = False) -> np.ndarray:
    """y = (S (.) W) x in float64, rounded once to fp32.  Returns M x N float32.

    int8 x: A[m, n, g] = sum_{k in g} W[n, k] x[m, k] is an exact integer and
    y[m, n] = sum_g S[n, g] * a[m, g] * A[m, n, g] (Sec. II-C).  bf16 x (given
    as raw bit patterns): the same sums with x widened exactly to float64.
    A per-tensor scale (group = 0) is one S for every (n, g); without
    activation scales (a = 1) it multiplies the full row sum once.
    """
    w = np.asarray(w, dtype=np.int8)
    n, k = w.shape
    if x_is_bf16_bits:
        xv = np.atleast_2d(bf16_bits_to_f64(np.asarray(x, dtype=np.uint16)))
    else:
        xv = np.atleast_2d(np.asarray(x, dtype=np.int64)).astype(np.float64)
    m = xv.shape[0]
    if xv.shape[1] != k:
        raise ValueError("x has the wrong length")
    wf = w.astype(np.float64)
    if group == 0 and xscale is None:
        s = fp16_bits_to_f64(np.asarray(scales_bits).reshape(-1))[0]
        return (s * (xv @ wf.T)).astype(np.float32)
    if k % 128:
        raise ValueError("group scales need K divisible by 128")
    g = k // 128
    # A[m, n, g]: one dot product per (row, group); exact for integer x.
    A = np.einsum("ngk,mgk->mng", wf.reshape(n, g, 128), xv.reshape(m, g, 128))
    if xscale is None:
        a = np.ones((m, g))
    else:
        a = np.asarray(xscale, dtype=np.float32).astype(np.float64).reshape(m, g)
    S = _expand_scales(scales_bits, n, k, group)                      # n x g
    y = np.einsum("ng,mg,mng->mn", S, a, A)
    return y.astype(np.float32)


def gemv_from_packed(p: Packed, x, xscale=None, x_is_bf16_bits=False, raw=False):
    """Decode a packed matrix with the oracle and run the dense definition."""
    if p.fmt == FMT_BITCOS:
        w, sc = bitcos_decode(p)
    elif p.fmt == FMT_TRIT5:
        w, sc = trit5_decode(p)
    elif p.fmt == FMT_BIT2:
        w, sc = bit2_decode(p)
    else:
        raise ValueError("unknown format")
    if raw:
        return dense_gemv_raw(w, x)
    return dense_gemv(w, sc, p.group, x, xscale, x_is_bf16_bits)


# ---------------------------------------------------------------------------
# Activation quantisation (Sec. II-C: int8 per group of 128)
# ---------------------------------------------------------------------------

def quantize_activations(x_bf16_bits: np.ndarray, group: int = 128) -> tuple[np.ndarray, np.ndarray]:
    """Per-group symmetric int8 quantisation, decisions taken in fp32.

    a = fp32(max|x| / 127) (a = 1 if the group is all zero);
    q = clamp(round_half_even(fp32(x / a)), -127, 127).
    Returns (q int8 [M, K], a float32 [M, K/group]).
    """
    x = np.atleast_2d(bf16_bits_to_f64(np.asarray(x_bf16_bits, dtype=np.uint16))).astype(np.float32)
    m, k = x.shape
    if k % group:
        raise ValueError("K must be a multiple of the group")
    xg = x.reshape(m, k // group, group)
    amax = np.max(np.abs(xg), axis=2)
    a = (amax / np.float32(127.0)).astype(np.float32)
    a = np.where(amax == 0, np.float32(1.0), a).astype(np.float32)
    q = np.rint((xg / a[:, :, None]).astype(np.float32))
    q = np.clip(q, -127, 127).astype(np.int8)
    return q.reshape(m, k), a


# ---------------------------------------------------------------------------
# Storage accounting (Sec. II-A Eq. (1), Sec. I, Table I)
# ---------------------------------------------------------------------------

def bpw_symbols_bitcos(z: float) -> float:
    """B(z) = 1 + (1 - z) = 2 - z bits per weight (Eq. (1))."""
    return 1.0 + (1.0 - z)


def bpw_trit5() -> float:
    """ceil(128 / 5) = 26 bytes per 128 weights (Sec. I)."""
    return math.ceil(128 / 5) * 8 / 128


def bpw_bit2() -> float:
    return 2.0


def scale_bits_per_weight(group: int) -> float:
    """One 16-bit scale per group of ``group`` weights (Table I's +scale)."""
    return 16.0 / group


def payload_bits(p: Packed) -> int:
    """Payload = format symbols + 16-bit scales (offsets/padding excluded)."""
    ns = p.num_scales()
    if p.fmt == FMT_BITCOS:
        return p.n * p.k + p.nnz + 16 * ns
    if p.fmt == FMT_TRIT5:
        return p.n * (p.k // 128) * TRIT5_BLOCK_BYTES * 8 + 16 * ns
    if p.fmt == FMT_BIT2:
        return 2 * p.n * p.k + 16 * ns
    raise ValueError("unknown format")


def bpw_payload(p: Packed) -> float:
    return payload_bits(p) / (p.n * p.k)


# ---------------------------------------------------------------------------
# Two-term CPU roofline (Sec. III-B1, Eqs. (5)-(6), Table II)
# ---------------------------------------------------------------------------

def roofline_bytes_per_32(z: float) -> float:
    """Bytes one 32-weight iteration reads: 4 (bitmap) + 4(1-z) (signs) + 0.5 (scale)."""
    return 4.0 + 4.0 * (1.0 - z) + 0.5


def roofline_cpu(z: float, beta: float, gamma: float) -> tuple[float, float, str]:
    """T = max(B/beta, gamma), e_bw = min(beta, B/gamma); returns (T, e_bw, bound)."""
    b = roofline_bytes_per_32(z)
    t = max(b / beta, gamma)
    e = min(beta, b / gamma)
    return t, e, ("memory" if b / gamma > beta else "instructions")
