"""GPU checks of aug_plan_upload (through the C ABI): the bytes arrive
unchanged, nothing past them is written, and pointers that are not pinned
host memory (source) or device memory (destination) are refused."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2512_04013_amd as aug  # noqa: E402
from tests.gpu_util import say  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

GUARD = 256


@pytest.mark.parametrize("nbytes", [1, 15, 16, 17, 4096 + 5, 121_024, (1 << 20) + 3, 3 << 20])
@pytest.mark.parametrize("offset", [0, 256])
def test_upload_copies_the_bytes_and_nothing_else(nbytes, offset):
    say(f"[plan upload] {nbytes} bytes at host offset {offset}")
    rng = np.random.default_rng(nbytes + offset)
    src = torch.empty(offset + nbytes, dtype=torch.uint8, pin_memory=True)
    src.numpy()[:] = rng.integers(0, 256, offset + nbytes, dtype=np.uint8)
    dst = torch.full((nbytes + GUARD,), 0xAB, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    aug.aug_plan_upload(src[offset:], dst, nbytes, stream=stream.cuda_stream)
    torch.cuda.synchronize()
    got = dst.cpu().numpy()
    assert np.array_equal(got[:nbytes], src.numpy()[offset:])
    assert np.all(got[nbytes:] == 0xAB)


def test_upload_then_kernels_on_the_same_stream_see_the_bytes():
    """Two uploads into one device buffer, each consumed by a device copy
    queued after it on the same stream, with no host synchronisation
    between: each consumer sees its own upload."""
    n = 200_000
    a = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    b = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    a.numpy()[:] = 1
    b.numpy()[:] = 2
    dst = torch.zeros(n, dtype=torch.uint8, device="cuda")
    seen = [torch.empty(n, dtype=torch.uint8, device="cuda") for _ in range(2)]
    s = torch.cuda.current_stream().cuda_stream
    aug.aug_plan_upload(a, dst, n, stream=s)
    seen[0].copy_(dst)
    aug.aug_plan_upload(b, dst, n, stream=s)
    seen[1].copy_(dst)
    torch.cuda.synchronize()
    assert bool((seen[0] == 1).all()) and bool((seen[1] == 2).all())


def test_upload_refuses_memory_of_the_wrong_kind():
    n = 4096
    pinned = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    pageable = torch.empty(n, dtype=torch.uint8)
    dev = torch.empty(n, dtype=torch.uint8, device="cuda")
    L = aug.lib()
    s = torch.cuda.current_stream().cuda_stream
    # source not page-locked, source on the device, destination on the host
    assert L.aug_plan_upload(pageable.data_ptr(), dev.data_ptr(), n, s) == aug.AUG_ERR_INVALID
    assert "pinned" in aug.aug_last_error()
    assert L.aug_plan_upload(dev.data_ptr(), dev.data_ptr(), n, s) == aug.AUG_ERR_INVALID
    assert L.aug_plan_upload(pinned.data_ptr(), pinned.data_ptr(), n, s) == aug.AUG_ERR_INVALID
    assert "device memory" in aug.aug_last_error()
    # a refused call leaves the runtime usable
    aug.aug_plan_upload(pinned, dev, n, stream=s)
    torch.cuda.synchronize()
