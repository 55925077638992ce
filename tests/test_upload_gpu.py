"""tg_plan_upload on the GPU through the C ABI: pinned host bytes arrive unchanged in
device memory, aligned and not, and nothing outside the destination is written."""
import ctypes

import numpy as np
import pytest

from gpu_helpers import say
from paper_2404_09267_amd import tg

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    tg.lib()
    return torch


@pytest.mark.parametrize("n", [1, 15, 16, 17, 4096, 40_003, (1 << 20) + 5])
def test_upload_sizes_and_offsets(torch, n):
    rng = np.random.default_rng(n)
    for so, do in ((0, 0), (1, 0), (0, 3), (5, 7), (16, 32)):
        say("upload", n, so, do)
        host = torch.empty(n + 64, dtype=torch.uint8, pin_memory=True)
        data = rng.integers(0, 256, n + 64, dtype=np.uint8)
        host.numpy()[:] = data
        dev = torch.full((n + 64,), 0xA5, dtype=torch.uint8, device="cuda")
        tg.plan_upload(host[so:so + n], dev[do:do + n])
        got = dev.cpu().numpy()
        np.testing.assert_array_equal(got[do:do + n], data[so:so + n])
        assert (got[:do] == 0xA5).all() and (got[do + n:] == 0xA5).all()


def test_upload_then_kernel_on_the_stream(torch):
    """The plan words reach the device before the next kernel on the stream reads them."""
    host = torch.empty(10_001, dtype=torch.int32, pin_memory=True)
    dev = torch.zeros(10_001, dtype=torch.int32, device="cuda")
    for k in range(3):
        host.numpy()[:] = np.arange(10_001, dtype=np.int32) * (k + 1)
        tg.plan_upload(host, dev)
        total = int(dev.to(torch.int64).sum().item())
        assert total == (k + 1) * 10_000 * 10_001 // 2


def test_upload_refuses_memory_that_is_not_pinned(torch):
    plain = np.arange(100, dtype=np.uint8)
    dev = torch.zeros(100, dtype=torch.uint8, device="cuda")
    rc = tg.lib().tg_plan_upload(ctypes.c_void_p(plain.ctypes.data), ctypes.c_void_p(dev.data_ptr()),
                                 100, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == tg.E_INVAL
    torch.cuda.synchronize()
    assert int(dev.sum().item()) == 0
