"""CPU tests of bench.py's host logic (no GPU: torch's graph calls are stubbed)."""

import contextlib
import os
import gc
import weakref

import pytest

torch = pytest.importorskip("torch")
import bench  # noqa: E402
import workloads as wl  # noqa: E402


class _FakeGraph:
    def replay(self):
        pass


@pytest.fixture
def fake_cuda(monkeypatch):
    c = torch.cuda
    monkeypatch.setattr(c, "Stream", lambda *a, **k: type("S", (), {"wait_stream": lambda self, o: None})())
    monkeypatch.setattr(c, "current_stream", lambda *a, **k: type("S", (), {"wait_stream": lambda self, o: None})())
    monkeypatch.setattr(c, "stream", lambda s: contextlib.nullcontext())
    monkeypatch.setattr(c, "graph", lambda g, **k: contextlib.nullcontext())
    monkeypatch.setattr(c, "synchronize", lambda *a, **k: None)
    monkeypatch.setattr(c, "CUDAGraph", _FakeGraph)


class _Tables:
    """Stands in for a batch's device tables: alive while referenced."""


def test_captured_graph_keeps_its_step_and_tables_alive(fake_cuda):
    """A graph's launches carry the device addresses of its batch tables and
    outputs; if the step (and its batches) were freed after capture, a replay
    would read whatever the allocator later put at those addresses."""
    tables = _Tables()
    calls = []

    def make():
        held = tables

        def step():
            calls.append(id(held))
        return step

    gs = [bench.capture(make()) for _ in range(2)]
    ref = weakref.ref(tables)
    del tables
    gc.collect()
    assert ref() is not None, "the captured step was dropped while its graph lives"
    assert len(calls) == 4  # one eager call and one captured call per graph
    del gs
    gc.collect()
    assert ref() is None


def test_device_copies_share_layouts_and_clone_blobs():
    class Blob:
        def __init__(self, tag):
            self.tag = tag

        def clone(self):
            return Blob(self.tag + "'")

    entries = [(0, 1, "spec", "L0", Blob("b0"), (0, 0, 8)), (1, 2, "spec", "L1", Blob("b1"), (1, 8, 8))]
    sets = bench.device_copies(entries, 3)
    assert len(sets) == 3 and sets[0] is entries
    for st in sets[1:]:
        assert [e[3] for e in st] == ["L0", "L1"]
        assert [e[4].tag for e in st] == ["b0'", "b1'"]
        assert all(a[4] is not b[4] for a, b in zip(st, entries))
        assert [e[5] for e in st] == [(0, 0, 8), (1, 8, 8)]


def test_supported_reports_baselines_without_a_long_row_kernel():
    """bf16 rows longer than 16384 have a BITCOS kernel at batch 1 (the
    small-batch kernel) but no five-trit or 2-bit kernel; int8 rows of that
    length have all three."""
    np = pytest.importorskip("numpy")
    api = pytest.importorskip("paper_2609_16338_amd.api")
    from paper_2609_16338_amd import _native as N

    rng = np.random.default_rng(5)
    k = 25600
    w = rng.integers(-1, 2, size=(3, k)).astype(np.int8)
    sc = np.full((3, k // 128), 0.01, np.float16)
    for fmt, bf16_ok in ((N.FMT_BITCOS, True), (N.FMT_TRIT5, False), (N.FMT_BIT2, False)):
        L, _ = api.plan_and_pack(fmt, w, sc, 128)
        entries = [(0, 6, None, L, None, (0, 0, k))]
        assert bench.supported(entries, "bf16", 1) is bf16_ok
        assert bench.supported(entries, "int8", 1)
        assert bench.supported(entries, "bf16", 4) is bf16_ok  # baselines at m > 1: batch-1 launches


def test_main_shadows_no_module_function():
    """A local of main() named like a module-level function (say `gamma`)
    would make main's call of that function fail before the function runs."""
    import inspect
    funcs = {n for n, v in vars(bench).items() if inspect.isfunction(v)}
    for fn in (bench.main,):
        assert not (set(fn.__code__.co_varnames) & funcs), set(fn.__code__.co_varnames) & funcs


def test_sample_rows_keep_first_and_last():
    for n in (1, 2, 5, 640, 25600):
        rows = bench.sample_rows(n, 3, 4)
        assert rows[0] == 0 and rows[-1] == n - 1
        assert len(set(rows.tolist())) == len(rows) <= max(bench.SAMPLE_ROWS, 1)
        assert np_all_in_range(rows, n)


def np_all_in_range(rows, n):
    return bool(((rows >= 0) & (rows < n)).all())


@pytest.mark.parametrize("group", [128, 0])
@pytest.mark.parametrize("kind", ["bf16", "int8"])
def test_self_check_reference_matches_the_oracle(group, kind):
    """bench.py's self-check reference (dense definition on sampled rows)
    agrees with the oracle's dense GEMV, and its error bars with the parity
    tests' bars."""
    np = pytest.importorskip("numpy")
    import oracle as O
    import workloads as wl
    from parity_checks import bf16_bound, group_bound

    n, k, m = 37, 640, 3
    w = wl.ternary(n, k, 0.45, wl.rng_for(70, group))
    ns = n * (k // 128) if group == 128 else 1
    sc = wl.fp16_uniform((ns,), 0.005, 0.05, wl.rng_for(71, group))
    rows = bench.sample_rows(n, 1, 2)
    sbits = sc.reshape(n, k // 128)[rows] if group == 128 else sc.reshape(1, 1)
    if kind == "bf16":
        xb = wl.act_bf16(m, k, wl.rng_for(72))
        ref = O.dense_gemv(w, sc, group, xb, x_is_bf16_bits=True)[:, rows]
        y, kbar, _ = bench.dense_rows(w[rows], sbits, group, bench.bf16_bits_to_f64(xb).reshape(m, k), None)
        bound = bf16_bound(w[rows], sc if group == 0 else sbits.reshape(-1), group, xb)
        assert np.allclose(kbar, bound, rtol=1e-12)
    else:
        q, a = O.quantize_activations(wl.act_bf16(m, k, wl.rng_for(73)))
        ref = O.dense_gemv(w, sc, group, q, a)[:, rows]
        y, _, gbar = bench.dense_rows(w[rows], sbits, group, q.astype(np.float64), a.astype(np.float64))
        bound = group_bound(w[rows], sc if group == 0 else sbits.reshape(-1), group, q, a)
        assert np.allclose(gbar, bound, rtol=1e-12)
    assert np.array_equal(y.astype(np.float32), ref)


def test_column_blocks_split_only_long_rows():
    assert bench.column_blocks(5120) == [(0, 5120)]
    assert bench.column_blocks(16384) == [(0, 16384)]
    # the Qwen3-32B-like down projection: five blocks of the hidden size
    assert bench.column_blocks(25600) == [(k0, 5120) for k0 in range(0, 25600, 5120)]
    for k in (16512, 20480, 32768, 49152):
        blocks = bench.column_blocks(k)
        assert sum(b for _, b in blocks) == k and all(b % 128 == 0 and b <= bench.KSPLIT_MAX for _, b in blocks)
        assert [k0 for k0, _ in blocks] == list(range(0, k, blocks[0][1]))


def test_stored_traffic_only_for_the_measured_launch():
    """A stored FETCH/WRITE measurement belongs to one launch (kernel, tile and
    GEMV count): a run of the same layer set on another kernel (the
    small-batch one at M > 1) or over other GEMVs must report traffic as
    unmeasured, not borrow another launch's figure."""
    path = bench.TRAFFIC_FILES["qwen3_32b_layers"][0]
    with open(path) as f:
        kv = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith("#"))
    launch = kv["launch"].strip()
    kernel, rest = launch.split("<", 1)
    other = "bitcos_mfma_kernel" if kernel != "bitcos_mfma_kernel" else "bitcos_fast_kernel"
    assert bench.stored_traffic("qwen3_32b_layers", f"{other}<{rest}") is None
    assert bench.stored_traffic("qwen3_32b_layers", launch.replace(" GEMVs", "0 GEMVs")) is None
    assert bench.stored_traffic("no_such_set", launch) is None
    if kv["kernel_source_hash"].strip() == bench.kernel_source_hash(kernel):
        assert bench.stored_traffic("qwen3_32b_layers", launch) == int(float(kv["traffic_bytes_per_launch"]))


def test_stored_valu_count_follows_the_sources(monkeypatch):
    """The stored SQ_INSTS_VALU count of the dominant launch is reported for
    that launch only, and only while its kernel sources hash as measured."""
    path = bench.COUNTER_FILES["qwen3_32b_layers"][0]
    with open(path) as f:
        kv = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith("#"))
    launch = kv["launch"].strip()
    assert bench.stored_valu("qwen3_32b_layers", launch.replace(" GEMVs", "0 GEMVs")) is None
    assert bench.stored_valu("no_such_set", launch) is None
    measured = kv["kernel_source_hash"].strip()
    monkeypatch.setattr(bench, "kernel_source_hash", lambda kernel="bitcos_fast_kernel": measured)
    assert bench.stored_valu("qwen3_32b_layers", launch) == int(float(kv["sq_insts_valu_per_launch"]))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda kernel="bitcos_fast_kernel": "0" * 16)
    assert bench.stored_valu("qwen3_32b_layers", launch) is None


def test_kernel_source_hash_ignores_comments_only(tmp_path, monkeypatch):
    """A stored measurement stays valid across comment edits, not code edits."""
    import shutil
    src = os.path.join(bench.ROOT, "paper_2609_16338_amd", "csrc")
    dst = tmp_path / "paper_2609_16338_amd" / "csrc"
    dst.mkdir(parents=True)
    for name in {n for names in bench.KERNEL_SOURCES.values() for n in names}:
        shutil.copy(os.path.join(src, name), dst / name)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = {k: bench.kernel_source_hash(k) for k in bench.KERNEL_SOURCES}
    f = dst / "tables.h"
    f.write_text(f.read_text() + "\n// a comment\n\n")
    assert {k: bench.kernel_source_hash(k) for k in bench.KERNEL_SOURCES} == h0
    # a code change in one kernel's own source leaves the others' measurements valid
    m = dst / "bitcos_mfma.h"
    m.write_text(m.read_text() + "constexpr int kUnusedForTheHashTest = 1;\n")
    assert bench.kernel_source_hash("bitcos_mfma_kernel") != h0["bitcos_mfma_kernel"]
    assert bench.kernel_source_hash("bitcos_fast_kernel") == h0["bitcos_fast_kernel"]
    f.write_text(f.read_text() + "constexpr int kUnusedForTheHashTest = 1;\n")
    assert all(bench.kernel_source_hash(k) != h0[k] for k in bench.KERNEL_SOURCES)


def test_sweep_points():
    """The sweep's shape and densities: the default 8192 x 8192 over the five
    densities and 0.95, or a given shape and list; a density of the sweep keeps
    its seed index, others get new ones."""
    n, k, pts = bench.sweep_points(bench.parse(["--sweep"]))
    assert (n, k) == (8192, 8192)
    assert pts == list(enumerate(wl.SWEEP_Z + (0.95,)))
    n, k, pts = bench.sweep_points(bench.parse(["--sweep", "--sweep-shape", "32768x16384", "--sweep-z", "0.42,0.6"]))
    assert (n, k) == (32768, 16384)
    assert pts == [(wl.SWEEP_Z.index(0.42), 0.42), (len(wl.SWEEP_Z) + 2, 0.6)]
    with pytest.raises(SystemExit):
        bench.sweep_points(bench.parse(["--sweep", "--sweep-shape", "100x100"]))

