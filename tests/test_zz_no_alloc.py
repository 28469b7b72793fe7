"""GPU test of bitcos_pack_device_noalloc, the packer entry point that
allocates nothing (its plan workspace is the library's fixed per-GPU array).

Two calls in a row through the C ABI, the second with a smaller matrix (and
another scale mode), each checked byte for byte against the existing
bitcos_plan_device + bitcos_pack_device pair with a caller workspace, and
against the oracle's serialised blob.  The limits are checked too: more rows
than the workspace holds, and a destination too small (the layout is still
reported).  Bar: identical bytes (byte work).
"""

import numpy as np
import pytest

import oracle as O
import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2609_16338_amd import _native as N  # noqa: E402
from paper_2609_16338_amd import api  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    N.lib()


def _oracle_blob(w, sc, group):
    blob, _ = O.serialize(O.bitcos_encode(w, sc, group, 1))
    return np.frombuffer(blob, dtype=np.uint8)


def _case(n, k, z, group, seed):
    w = wl.ternary(n, k, z, wl.rng_for(800, seed))
    ns = n * (k // 128) if group == 128 else 1
    sc = wl.fp16_uniform((ns,), 0.005, 0.05, wl.rng_for(801, seed))
    return w, sc


def test_noalloc_packer_matches_the_workspace_packer_twice():
    cases = [(700, 2560, 0.45, 128, 1), (37, 640, 0.3, 0, 2)]  # second call smaller
    for n, k, z, group, seed in cases:
        w, sc = _case(n, k, z, group, seed)
        wd = torch.from_numpy(w).cuda()
        sd = torch.from_numpy(sc.view(np.int16)).cuda()
        L_ref, blob_ref = api.bitcos_pack_device(wd, sd, group)
        dst = torch.full((L_ref.total_bytes + 512,), 0xA5, dtype=torch.uint8, device="cuda")
        L = api.bitcos_pack_device_noalloc(wd, sd, dst, group)
        torch.cuda.synchronize()
        assert L.total_bytes == L_ref.total_bytes and L.nnz == L_ref.nnz
        assert bytes(L) == bytes(L_ref)
        got = dst.cpu().numpy()
        ref = blob_ref.cpu().numpy()
        assert np.array_equal(got[:L.total_bytes], ref)
        assert np.all(got[L.total_bytes:] == 0xA5), "wrote past the blob"
        assert np.array_equal(got[:L.total_bytes], _oracle_blob(w, sc, group))


def test_noalloc_packer_limits():
    w, sc = _case(64, 256, 0.4, 128, 3)
    wd = torch.from_numpy(w).cuda()
    sd = torch.from_numpy(sc.view(np.int16)).cuda()
    small = torch.zeros(256, dtype=torch.uint8, device="cuda")
    with pytest.raises(N.BitcosError) as e:
        api.bitcos_pack_device_noalloc(wd, sd, small, 128)
    assert e.value.status == N.E_SPACE
    L_want, _ = api.plan_and_pack(N.FMT_BITCOS, w, sc, 128)
    assert e.value.layout.total_bytes == L_want.total_bytes  # the size needed is reported
    assert np.all(small.cpu().numpy() == 0)
    # More rows than the fixed workspace holds: rejected before any device work.
    n_big = N.NOALLOC_MAX_ROWS + 1
    L = N.Layout()
    st = N.lib().bitcos_pack_device_noalloc(wd.data_ptr(), sd.data_ptr(), n_big, 128, 0, 0, L,
                                            small.data_ptr(), small.numel(), None)
    assert st == N.E_SPACE
