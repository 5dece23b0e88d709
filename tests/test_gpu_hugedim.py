"""One run whose rows hold more floats than a 32-bit index reaches (marked
gpu): D = 2^31 + 5, N = 2, about 100 GB of device memory in all.

Windows of dims that straddle element 2^31, the ragged end and the start are
compared with the oracle, which computes any window of the stream on its own:
the materialised members (m = 0, so x = +-sigma*z; bound sigma * 2.6e-6, the
normals' error), the fitness against an fp64 sum of the materialised members
on the device (1e-5 relative), the gradient against the oracle's from the
GPU's shaped weights (|w| 2.6e-6 / (N sigma) per dim) and the Adam step
bit-exact given the kernel's gradient.
"""
import numpy as np
import pytest
import torch

from inputs import to_oracle
from oracle import oracle as O

pytestmark = pytest.mark.gpu

DZ = 2.6e-6


def test_dims_beyond_32_bit_indices():
    import paper_2212_04180_amd as P
    free, _ = torch.cuda.mem_get_info()
    if free < 120 * (1 << 30):
        pytest.skip("needs about 100 GB of free device memory")
    D = (1 << 31) + 5
    sigma = 0.5
    cfg = P.ESConfig(num_dims=D, popsize=2, num_runs=1, sigma=sigma, lr=0.1, seed=9, init=P.INIT_ZERO,
                     problem=P.PROB_SPHERE, flags=P.FLAG_KEEP_GRAD)
    oc = to_oracle(cfg)
    windows = [(0, 8), ((1 << 31) - 8, 12), (D - 13, 13)]  # the second straddles element 2^31
    es = P.ES(cfg)
    x = es.ask(materialize=True)
    f = es.eval()
    torch.cuda.synchronize()
    ch = 1 << 28
    for j in range(2):
        ref = sum(float((x[0, j, s:s + ch].double() ** 2).sum()) for s in range(0, D, ch))
        got = float(f[0, j])
        assert abs(got - ref) <= 1e-5 * ref, (j, got, ref)
    for d0, nd in windows:
        z = O.noise(oc, 0, 0, 0, d0, nd).astype(np.float64)
        xp = x[0, 0, d0:d0 + nd].cpu().numpy()
        xm = x[0, 1, d0:d0 + nd].cpu().numpy()
        np.testing.assert_array_equal(xm, -xp)
        assert np.all(np.abs(xp - sigma * z) <= sigma * DZ + 1e-7 * np.abs(xp)), (d0, xp, sigma * z)
    del x
    torch.cuda.empty_cache()
    es.tell(f)
    y = es.shaped()[0][0].cpu().numpy()
    g = es.grad()
    st = es.get_state()
    torch.cuda.synchronize()
    bound = np.sum(np.abs(y)) * DZ / (2 * sigma)
    for d0, nd in windows:
        gw = g[0, d0:d0 + nd].cpu().numpy()
        gr = O.grad(oc, 0, 0, y, d0, nd)
        assert np.all(np.abs(gw - gr) <= bound + 1e-6 * np.abs(gr)), (d0, gw, gr)
        zero = np.zeros(nd, np.float32)
        m, m1, v = O.adam(oc, 0, gw, zero, zero, zero)
        np.testing.assert_array_equal(st["m"][0, d0:d0 + nd].cpu().numpy(), m)
        np.testing.assert_array_equal(st["m1"][0, d0:d0 + nd].cpu().numpy(), m1)
        np.testing.assert_array_equal(st["v"][0, d0:d0 + nd].cpu().numpy(), v)
    assert st["t"] == 1
