"""Multi-layer error correction (Sec. 3.3.3) on the GPU (quantize_net, which
chains qcnn_pq_kmeans, qcnn_ec_conv / qcnn_ec_fc and the PQ forward) against
the oracle chain (oracle/ec_network.py) on a conv -> pool -> conv -> FC stack.
The original network's responses T are an input of the method; both sides
take the oracle's (float64 dense layers rounded to fp32).

Layer 1 sees identical inputs on both sides; later layers see the quantized
network's activations, which the GPU's fp32 forward and the oracle's float64
forward (rounded to fp32) produce to within the forward's bound, so the
inputs, sub-codebooks and objectives agree to that accuracy and the codes
are equal (no near ties on these inputs).
"""
import os
import sys

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

sys.path.insert(0, os.path.dirname(__file__))


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def to_dev(specs, dev):
    out = []
    for s in specs:
        d = dict(s)
        for k in ("W", "D0", "bias"):
            if d.get(k) is not None:
                d[k] = torch.from_numpy(np.ascontiguousarray(d[k])).to(dev)
        out.append(d)
    return out


@pytest.mark.parametrize("seed,lossless", [(5, False), (6, False), (7, True)])
def test_network_matches_oracle(dev, seed, lossless):
    import pin_battery
    from oracle import ec_network
    from paper_1512_06473_amd import quantize_net
    x, specs = pin_battery.small_network(np.random.Generator(np.random.PCG64(seed)), lossless)
    print("ec_network seed", seed, flush=True)
    rec = []
    # the original network's responses are the caller's: the oracle's here
    targets = [None if t is None else torch.from_numpy(t).to(dev) for t in ec_network.original_responses(x, specs)]
    got = quantize_net.quantize_network(torch.from_numpy(x).to(dev), to_dev(specs, dev), targets, sweeps=1, inner=1,
                                        kmeans_iters=2, record=rec)
    torch.cuda.synchronize()
    ref = ec_network.quantize_network(x, specs, sweeps=1, inner=1, kmeans_iters=2)
    li = 0
    for g, r in zip(got, ref):
        if r is None:
            assert g is None
            continue
        D, codes, hist, S, T = r
        Sg, Tg = rec[li]
        li += 1
        assert np.allclose(Sg.cpu().numpy(), S, rtol=1e-5, atol=1e-6)
        assert np.allclose(Tg.cpu().numpy(), T, rtol=1e-6, atol=1e-6)
        assert np.array_equal(g["codes"].cpu().numpy(), codes)
        scale = max(float(np.abs(D).max()), 1e-30)
        assert np.allclose(g["D"].cpu().numpy(), D, rtol=1e-4, atol=1e-6 * scale)
        o = g["objective"].cpu().numpy()
        energy = float(np.sum(T.astype(np.float64) ** 2))  # errors are relative to the responses' size
        assert np.allclose(o, hist, rtol=1e-4, atol=1e-10 * energy)
        if lossless:
            assert o[-1] <= 1e-10 * energy
