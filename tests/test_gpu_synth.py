"""The seeded input generators: the device fills (what the GPU runs read) and
the host fills (what the oracle reads) give the same bits at every index,
for any starting index, length and key.  Parity failures then point at the
method, never at its inputs."""
import numpy as np
import pytest

import synth
from synth import configs as C

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.mark.parametrize("n,idx0,seed,step,per_mille,factor", [
    (1, 0, 0, 0, 0, 1.0),
    (1001, 0, 0, 3, 0, 1.0),
    (4099, 12345, 7, 1, 10, 100.0),
    (70001, 3, 2, 9, 1, 1000.0),
])
def test_normal_fill_device_equals_host(torch_cuda, n, idx0, seed, step, per_mille, factor):
    torch = torch_cuda
    k = synth.key(seed, C.STREAM_G, step)
    ks = C.ksigma(1e-3)
    dev = torch.empty(n, dtype=torch.float32, device="cuda")
    synth.normal_dev(dev, idx0, k, ks, per_mille, factor)
    host = synth.normal_host(n, idx0, k, ks, per_mille, factor)
    assert np.array_equal(dev.cpu().numpy().view(np.uint32), host.view(np.uint32))


@pytest.mark.parametrize("n,idx0,w", [(1, 0, 1), (257, 0, 3), (5003, 999, 127)])
def test_bits_and_scales_fill_device_equals_host(torch_cuda, n, idx0, w):
    torch = torch_cuda
    kb = synth.key(w, C.STREAM_BITS, 2)
    bdev = torch.empty(n, dtype=torch.int64, device="cuda")
    synth.bits_dev(bdev, idx0, kb)
    assert np.array_equal(bdev.cpu().numpy().view(np.uint64),
                          synth.bits_host(n, idx0, kb).view(np.uint64))
    ks = synth.key(w, C.STREAM_SCALES, 2)
    sdev = torch.empty(n, dtype=torch.float32, device="cuda")
    synth.scales_dev(sdev, idx0, ks, 3.6e-8)
    assert np.array_equal(sdev.cpu().numpy().view(np.uint32),
                          synth.scales_host(n, idx0, ks, 3.6e-8).view(np.uint32))
