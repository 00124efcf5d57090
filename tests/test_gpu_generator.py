"""The GPU fill kernels of the workload generator write the same bits as
the host generator (so the GPU path and the oracle read identical inputs)."""
import numpy as np
import pytest
import torch

import workload as wl
from workload import device as wd

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n,seed,stream,offset,std", [
    (1000003, 3, wl._wstream(5, wl.W_G), 0, 0.02),
    (4096, 11, wl._kvstream(63, 17, 1), 123456789, 1.0),
    (77, 2**40 + 5, 0xFFFFFFFF, 2**33, 0.5),
])
def test_normal_fill_bit_identical(n, seed, stream, offset, std):
    for bf16 in (True, False):
        host = np.empty(n, np.uint16 if bf16 else np.float32)
        fn = wl.lib().wl_fill_normal_bf16 if bf16 else wl.lib().wl_fill_normal_f32
        fn(host.ctypes.data, n, seed, stream, offset, std)
        dev = torch.empty(n, dtype=torch.int16 if bf16 else torch.float32, device="cuda")
        wd.gpu_fill_normal(dev, seed, stream, offset, std)
        got = dev.cpu().numpy()
        assert np.array_equal(got.view(host.dtype), host)


def test_uniform_fill_bit_identical():
    n = 300001
    for bf16 in (True, False):
        host = np.empty(n, np.uint16 if bf16 else np.float32)
        fn = wl.lib().wl_fill_uniform_bf16 if bf16 else wl.lib().wl_fill_uniform_f32
        fn(host.ctypes.data, n, 9, 1234, 55, 0.5, 1.5)
        dev = torch.empty(n, dtype=torch.int16 if bf16 else torch.float32, device="cuda")
        wd.gpu_fill_uniform(dev, 9, 1234, 55, 0.5, 1.5)
        assert np.array_equal(dev.cpu().numpy().view(host.dtype), host)


def test_device_weights_match_host_weights():
    m = wl.MODELS["tiny-bf16"]
    dw = wd.DeviceWeights(m, 5, gamma="uniform")
    for kind in (wl.W_Q, wl.W_D, wl.N_1, wl.N_K):
        for l in range(m.n_layers):
            host = wl.new_weight(m, 5, l, kind, "uniform")
            assert np.array_equal(dw.layer[kind][l].cpu().numpy().view(np.uint16), host)
    assert np.array_equal(dw.glob[wl.LM_HEAD].cpu().numpy().view(np.uint16),
                          wl.new_weight(m, 5, -1, wl.LM_HEAD))
