"""CPU tests of bench.py's host logic (no GPU: torch's graph calls are stubbed)."""

import contextlib
import gc
import weakref

import pytest

torch = pytest.importorskip("torch")
import bench  # noqa: E402


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

    entries = [(0, 1, "spec", "L0", Blob("b0")), (1, 2, "spec", "L1", Blob("b1"))]
    sets = bench.device_copies(entries, 3)
    assert len(sets) == 3 and sets[0] is entries
    for st in sets[1:]:
        assert [e[3] for e in st] == ["L0", "L1"]
        assert [e[4].tag for e in st] == ["b0'", "b1'"]
        assert all(a[4] is not b[4] for a, b in zip(st, entries))
