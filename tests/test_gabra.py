"""The library's GABRA (host C++, rat3d_gabra) against the oracle
(oracle/gabra.py): both follow the paper's Algorithms 1-3 with the same
readings and draw from the same SplitMix64 sequence, so the allocation, the
profit (bit for bit) and the counters must be identical; plus argument
validation.  Host code: runs without a GPU."""
import numpy as np
import pytest

from oracle import gabra as G
from paper_2104_05035_amd import rat3d as R


def _instance(seed):
    rng = np.random.default_rng(1000 + seed)
    n, m = int(rng.integers(1, 13)), int(rng.integers(1, 7))
    p = rng.uniform(0.5, 20.0, n)
    d = rng.uniform(0.5, 1.5, m)
    d = np.maximum(d / d.sum() * p.sum() * rng.uniform(1.05, 2.0), p.max())
    return list(map(float, p)), list(map(float, d)), bool(rng.integers(0, 2)) and n >= m


@pytest.mark.parametrize("seed", range(24))
def test_library_matches_oracle(seed):
    p, d, every = _instance(seed)
    kw = dict(population=int(4 + seed % 9), generations=int(50 + 37 * seed), seed=seed * 7919,
              every_gpu=every, crossover_p=(0.8, 1.0, 0.0, 0.5)[seed % 4])
    try:
        zo, fo, so = G.gabra(p, d, **kw)
    except ValueError:
        with pytest.raises(R.Rat3dError) as e:
            R.rat3d_gabra(p, d, **kw)
        assert e.value.status == R.EINVAL
        return
    z, f, st = R.rat3d_gabra(p, d, **kw)
    assert z == zo and f == fo and st == so


def test_network_stages_to_gpus():
    """The stem and the three stages of the full network, loaded by their conv
    work per step of 8 volumes (45, 527, 264, 135 GFLOP), onto three GPUs of
    unequal capacity (GFLOP per step they may take): the library's allocation
    is feasible and reaches the exact optimum."""
    p = [45.0, 527.0, 264.0, 135.0]
    d = [600.0, 400.0, 300.0]
    best, fb = G.brute_force(p, d)
    z, f, _ = R.rat3d_gabra(p, d, population=20, generations=400, seed=2)
    assert f == pytest.approx(fb, rel=1e-12) and G.feasible(z, p, d)


@pytest.mark.parametrize("kw,args", [
    (dict(), ([1.0, -1.0], [2.0])), (dict(), ([1.0], [0.0])), (dict(population=1), ([1.0], [2.0])),
    (dict(crossover_p=1.5), ([1.0], [2.0])), (dict(), ([], [2.0])), (dict(), ([1.0], [])),
    (dict(), ([float("nan")], [2.0])), (dict(), ([3.0, 3.0], [2.0, 2.0])),
])
def test_validation(kw, args):
    with pytest.raises(R.Rat3dError) as e:
        R.rat3d_gabra(*args, **kw)
    assert e.value.status == R.EINVAL
