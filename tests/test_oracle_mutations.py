"""Mutation check of the oracle's pins.

Each case plants one plausible slip in a copy of the oracle -- a dropped
term, a flipped sign or polarity, an off-by-one rank or index, a transposed
operand, a wrong bit order -- and runs the pin tests (test_oracle_pins.py)
against that copy in a separate process.  Every slip must make at least one
pin fail: a slip the pins cannot see would leave the oracle unchecked there.

The copy lives in a temporary tree (oracle/, the pin tests with their
conftest, golden files and helpers, and the input generators), so the real
oracle is never modified and the copy's conftest puts the mutated oracle
first on the import path.
"""

import os
import shutil
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle", "bitcos_oracle.py")

# (name, text in bitcos_oracle.py, replacement): each a single slip.
MUTATIONS = [
    ("pdep takes the source bit from the mask index",
     "            if (a >> k) & 1:\n                dst |= 1 << m",
     "            if (a >> m) & 1:\n                dst |= 1 << m"),
    ("Eq. (2) with +2n instead of -2n", "    return p - 2 * n", "    return p + 2 * n"),
    ("table rank counts the row itself",
     "        r_i = sum((m >> j) & 1 for j in range(i))",
     "        r_i = sum((m >> j) & 1 for j in range(i + 1))"),
    ("table sign polarity flipped",
     "        codes.append(-1 if (s >> r_i) & 1 else +1)",
     "        codes.append(+1 if (s >> r_i) & 1 else -1)"),
    ("table cursor advance dropped", "    return tuple(codes), popcount(m)", "    return tuple(codes), 4"),
    ("sign stream polarity flipped",
     "    negative = (flat[flat != 0] < 0).astype(np.uint8)",
     "    negative = (flat[flat != 0] > 0).astype(np.uint8)"),
    ("bitmap bit order MSB first",
     '    return np.packbits(padded, bitorder="little").view("<u4")',
     '    return np.packbits(padded, bitorder="big").view("<u4")'),
    ("unit offsets count one unit late",
     "        off[u] = off[u - 1] + per_row[(u - 1) * unit_rows: min(u * unit_rows, n)].sum()",
     "        off[u] = off[u - 1] + per_row[u * unit_rows: min((u + 1) * unit_rows, n)].sum()"),
    ("dense GEMV drops the group scale",
     '    y = np.einsum("ng,mg,mng->mn", S, a, A)',
     '    y = np.einsum("mg,mng->mn", a, A)'),
    ("dense GEMV drops the activation scale",
     '    y = np.einsum("ng,mg,mng->mn", S, a, A)',
     '    y = np.einsum("ng,mng->mn", S, A)'),
    ("dense GEMV transposes the group sums",
     '    A = np.einsum("ngk,mgk->mng", wf.reshape(n, g, 128), xv.reshape(m, g, 128))',
     '    A = np.einsum("ngk,mgk->mng", wf.reshape(n, 128, g).transpose(0, 2, 1), xv.reshape(m, g, 128))'),
    ("raw GEMV uses W instead of W transposed",
     "    return x64 @ w64.T",
     "    return (w64 @ x64.T).T[:, ::-1]"),
    ("quantiser divides by 128", "    a = (amax / np.float32(127.0)).astype(np.float32)",
     "    a = (amax / np.float32(128.0)).astype(np.float32)"),
    ("quantiser rounds half away from zero",
     "    q = np.rint((xg / a[:, :, None]).astype(np.float32))",
     "    q = np.trunc((xg / a[:, :, None]).astype(np.float32) + np.copysign(0.5, xg))"),
    ("Eq. (1) with 2 + z", "    return 1.0 + (1.0 - z)", "    return 1.0 + (1.0 + z)"),
    ("five-trit rate with 25 bytes", "    return math.ceil(128 / 5) * 8 / 128", "    return (128 // 5) * 8 / 128"),
    ("payload drops the scales", "        return p.n * p.k + p.nnz + 16 * ns", "        return p.n * p.k + p.nnz"),
    ("roofline sign bytes use z instead of 1 - z", "    return 4.0 + 4.0 * (1.0 - z) + 0.5",
     "    return 4.0 + 4.0 * z + 0.5"),
    ("roofline takes the smaller term", "    t = max(b / beta, gamma)", "    t = min(b / beta, gamma)"),
    ("five-trit digit weights 3**(t+1)", "            val += d * 3 ** t", "            val += d * 3 ** (t + 1)"),
    ("2-bit fields swapped", "            word |= c[:, :, t, b] << np.uint32(8 * b + 2 * t)",
     "            word |= c[:, :, t, b] << np.uint32(8 * t + 2 * b)"),
]


def _tree_with(mutated_source):
    d = tempfile.mkdtemp(prefix="oracle_mut_")
    os.makedirs(os.path.join(d, "oracle"))
    shutil.copy(os.path.join(ROOT, "oracle", "__init__.py"), os.path.join(d, "oracle", "__init__.py"))
    with open(os.path.join(d, "oracle", "bitcos_oracle.py"), "w") as f:
        f.write(mutated_source)
    shutil.copy(os.path.join(ROOT, "workloads.py"), d)
    os.makedirs(os.path.join(d, "tests"))
    for name in ("conftest.py", "test_oracle_pins.py"):
        shutil.copy(os.path.join(ROOT, "tests", name), os.path.join(d, "tests", name))
    for sub in ("golden", "helpers"):
        shutil.copytree(os.path.join(ROOT, "tests", sub), os.path.join(d, "tests", sub))
    return d


def _run_pins(tree):
    env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1")
    p = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(tree, "tests", "test_oracle_pins.py")],
                       cwd=tree, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=600)
    return p.returncode, p.stdout


def test_unmutated_copy_passes():
    """The copied tree itself passes its pins (so a failure below is the slip's)."""
    with open(ORACLE) as f:
        src = f.read()
    tree = _tree_with(src)
    try:
        rc, out = _run_pins(tree)
        assert rc == 0, out[-2000:]
    finally:
        shutil.rmtree(tree, ignore_errors=True)


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_pins_catch_the_slip(name, old, new):
    with open(ORACLE) as f:
        src = f.read()
    assert src.count(old) == 1, f"mutation site not found once: {name}"
    tree = _tree_with(src.replace(old, new))
    try:
        rc, out = _run_pins(tree)
        assert rc != 0, f"no pin caught: {name}"
        assert "failed" in out or "error" in out.lower(), out[-2000:]
    finally:
        shutil.rmtree(tree, ignore_errors=True)
