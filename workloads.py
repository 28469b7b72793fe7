"""Seeded synthetic inputs for the BITCOS GEMV: ternary matrices, scales, activations.

This module is shared by the test suite, the benchmark and the smoke check.
It produces *inputs* only and holds none of the method's arithmetic (no
packing, no decoding, no GEMV).  Every array is a deterministic function of a
seed, so the HIP path and the CPU oracle can be fed identical data.

Recipe (the paper's checkpoints are not available; its GEMV benchmark is
synthetic too):
* ternary weights: every element is zero with probability z, otherwise +1 or
  -1 with equal probability, independently (``ternary``).  A 16-bit uniform
  draw u per element (Philox, four draws per raw 64-bit output) decides both:
  zero iff u < T with T = 2 * round(z * 32768), and the sign is the parity of
  u (odd = -1), exactly balanced on [T, 65536) because T is even.  So the
  realised probability of a zero is T / 65536 (within 2**-16 of z).
  ``row_z`` gives every row its own density (the non-iid Qwen3-32B-like set).
  ``ternary_exact`` places an exact number of zeros (for the z = 0.375
  crossover).
* scales: fp16 of a uniform draw in [lo, hi] (returned as uint16 bit patterns).
* activations: int8 uniform integers in [-127, 127]; bf16 from N(0, 1) rounded
  to nearest-even (returned as uint16 bit patterns).
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

# ---------------------------------------------------------------------------
# Generators
# ---------------------------------------------------------------------------


def rng_for(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(np.random.SeedSequence(list(key))))


def _threshold(z: float) -> int:
    return 2 * int(round(min(max(float(z), 0.0), 1.0) * 32768))


def _u16(rng: np.random.Generator, count: int) -> np.ndarray:
    raw = rng.bit_generator.random_raw((count + 3) // 4)
    return raw.view(np.uint16)[:count]


def ternary(n: int, k: int, z: float, seed, row_z: np.ndarray | None = None) -> np.ndarray:
    """N x K int8 in {-1, 0, +1}: zero with probability z (or row_z[n]), signs balanced."""
    rng = seed if isinstance(seed, np.random.Generator) else rng_for(*np.atleast_1d(seed).tolist())
    u = _u16(rng, n * k).reshape(n, k)
    if row_z is None:
        table = np.where(np.arange(65536) & 1, np.int8(-1), np.int8(1)).astype(np.int8)
        table[: _threshold(z)] = 0
        return table[u]
    thr = np.array([_threshold(v) for v in np.asarray(row_z, dtype=np.float64)], dtype=np.int32)
    w = np.where(u & 1, np.int8(-1), np.int8(1)).astype(np.int8)
    w[u.astype(np.int32) < thr[:, None]] = 0
    return w


def ternary_exact(n: int, k: int, nzeros: int, seed) -> np.ndarray:
    """N x K ternary with exactly ``nzeros`` zeros at random positions, signs balanced."""
    rng = seed if isinstance(seed, np.random.Generator) else rng_for(*np.atleast_1d(seed).tolist())
    flat = np.where(rng.integers(0, 2, size=n * k) == 1, -1, 1).astype(np.int8)
    pos = rng.permutation(n * k)[:nzeros]
    flat[pos] = 0
    return flat.reshape(n, k)


def fp16_uniform(shape, lo: float, hi: float, seed) -> np.ndarray:
    rng = seed if isinstance(seed, np.random.Generator) else rng_for(*np.atleast_1d(seed).tolist())
    return rng.uniform(lo, hi, size=shape).astype(np.float16).view(np.uint16)


def act_int8(m: int, k: int, seed) -> np.ndarray:
    rng = seed if isinstance(seed, np.random.Generator) else rng_for(*np.atleast_1d(seed).tolist())
    return rng.integers(-127, 128, size=(m, k), dtype=np.int16).astype(np.int8)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to the nearest bfloat16 (ties to even); returns uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16)


def act_bf16(m: int, k: int, seed) -> np.ndarray:
    rng = seed if isinstance(seed, np.random.Generator) else rng_for(*np.atleast_1d(seed).tolist())
    return f32_to_bf16_bits(rng.standard_normal(size=(m, k)).astype(np.float32))


# ---------------------------------------------------------------------------
# Workload registry (the five configurations the GEMV is measured on)
# ---------------------------------------------------------------------------


@dataclass(frozen=True)
class MatrixSpec:
    name: str
    n: int            # output rows
    k: int            # reduction length
    z: float          # zero density (mean, for per-row densities)
    group: int        # 128 or 0 (one scale per tensor)
    scale_lo: float
    scale_hi: float
    row_z: tuple | None = None   # (lo, hi): per-row density drawn uniform in [lo, hi]


@dataclass(frozen=True)
class Workload:
    cid: int
    name: str
    layers: int
    matrices: tuple        # of MatrixSpec
    act: tuple             # activation kinds: "int8", "bf16"
    batch: tuple = (1,)


def _layer(h: int, kv: int, ffn: int, z: float, group: int, lo: float, hi: float, row_z=None):
    spec = lambda nm, n, k: MatrixSpec(nm, n, k, z, group, lo, hi, row_z)  # noqa: E731
    return (spec("q", h, h), spec("k", kv, h), spec("v", kv, h), spec("o", h, h),
            spec("gate", ffn, h), spec("up", ffn, h), spec("down", h, ffn))


WORKLOADS = {
    # Smallest instance: one 256 x 1024 matrix, z = 0.5, g128 scales, int8 x.
    "single_256x1024": Workload(1, "single_256x1024", 1,
                                (MatrixSpec("w", 256, 1024, 0.50, 128, 0.01, 0.1),), ("int8",)),
    # BitNet-2B-like decode layer set: 30 layers, hidden 2560, FFN 6912, k/v 640.
    "bitnet2b_layers": Workload(2, "bitnet2b_layers", 30,
                                _layer(2560, 640, 6912, 0.42, 0, 0.01, 0.1), ("bf16", "int8")),
    # Qwen3-8B-like: 36 layers, hidden 4096, FFN 12288, k/v 1024, g128.
    "qwen3_8b_layers": Workload(3, "qwen3_8b_layers", 36,
                                _layer(4096, 1024, 12288, 0.467, 128, 0.005, 0.05), ("bf16", "int8")),
    # Qwen3-32B-like: 64 layers, hidden 5120, FFN 25600, k/v 1024, per-row z.
    "qwen3_32b_layers": Workload(5, "qwen3_32b_layers", 64,
                                 _layer(5120, 1024, 25600, 0.45, 128, 0.005, 0.05, (0.30, 0.60)),
                                 ("int8", "bf16"), (1, 4, 16)),
}

SWEEP_Z = (0.30, 0.375, 0.42, 0.467, 0.515)


def sweep_spec(z: float, n: int = 8192, k: int = 8192) -> MatrixSpec:
    """One matrix of the zero-density sweep (g128, int8 x): 8192 x 8192, or
    another shape such as the paper's 32768 x 16384 sweep matrix."""
    return MatrixSpec(f"sweep_z{z}", n, k, z, 128, 0.01, 0.1)


def matrix_inputs(cid: int, layer: int, midx: int, spec: MatrixSpec):
    """(W, scales) for matrix ``midx`` of ``layer`` of workload ``cid``."""
    rng = rng_for(cid, layer, midx, 0)
    row_z = None
    if spec.row_z is not None:
        row_z = rng.uniform(spec.row_z[0], spec.row_z[1], size=spec.n)
    w = ternary(spec.n, spec.k, spec.z, rng, row_z=row_z)
    ns = spec.n * (spec.k // 128) if spec.group == 128 else 1
    sc = fp16_uniform((ns,), spec.scale_lo, spec.scale_hi, rng_for(cid, layer, midx, 1))
    return w, sc


def activation_inputs(cid: int, kind: str, m: int, k: int, salt: int = 0):
    if kind == "int8":
        return act_int8(m, k, rng_for(cid, 1000 + salt, k, 2))
    if kind == "bf16":
        return act_bf16(m, k, rng_for(cid, 1000 + salt, k, 3))
    raise ValueError(kind)
