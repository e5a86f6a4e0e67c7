"""Runtime behaviour of the library on the device (no numerics here).

The library's stream-ordered workspaces come from a memory pool it creates
itself: after conv and FC calls that needed workspaces, the device's default
pool still has its own release threshold (0 unless the application changed
it), so the library leaves process-wide state alone.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_1512_06473_amd import api
from paper_1512_06473_amd import workloads as wl

pytestmark = pytest.mark.gpu

RELEASE_THRESHOLD = 0x4  # hipMemPoolAttrReleaseThreshold


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def default_pool_threshold(device_index):
    hip = ctypes.CDLL("libamdhip64.so")
    pool = ctypes.c_void_p()
    assert hip.hipDeviceGetDefaultMemPool(ctypes.byref(pool), ctypes.c_int(device_index)) == 0
    val = ctypes.c_uint64(12345)
    assert hip.hipMemPoolGetAttribute(pool, ctypes.c_int(RELEASE_THRESHOLD), ctypes.byref(val)) == 0
    return val.value


def test_default_pool_left_alone(dev):
    before = default_pool_threshold(dev.index or 0)
    rng = np.random.Generator(np.random.PCG64(4))
    # a split conv layer (partial sums in the workspace) and a tiled FC layer
    x, D, codes = wl.random_conv(rng, 8, 256, 13, 13, 384, 3, 1, 1, 4, 128)
    y = api.conv_forward(torch.from_numpy(x).to(dev), torch.from_numpy(D).to(dev), torch.from_numpy(codes).to(dev),
                         1, 1)
    xf, Df, cf = wl.random_fc(rng, 64, 1024, 512, 4, 32)
    z = api.fc_forward(torch.from_numpy(xf).to(dev), torch.from_numpy(Df).to(dev), torch.from_numpy(cf).to(dev))
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y).all()) and bool(torch.isfinite(z).all())
    after = default_pool_threshold(dev.index or 0)
    assert after == before, (before, after)
    assert after != 2 ** 64 - 1
