"""The GPU build of the input generators gives the same graphs as the CPU
build (byte for byte after sort/dedup)."""
import numpy as np
import pytest

from paper_2607_02603_amd import inputs

pytestmark = pytest.mark.gpu


def _same(a, b):
    b = b.to_numpy()
    assert a.n == b.n
    assert np.array_equal(a.row_ptr.astype(np.uint64), b.row_ptr.astype(np.uint64))
    assert np.array_equal(a.col.astype(np.uint32), b.col.view(np.uint32))


@pytest.mark.parametrize("scale,ef,seed", [(10, 16, 0), (14, 16, 3), (16, 8, 1)])
def test_rmat_gpu_equals_cpu(scale, ef, seed, gpu_device):
    _same(inputs.rmat(scale, ef, seed=seed), inputs.rmat(scale, ef, seed=seed,
                                                         device="cuda"))


@pytest.mark.parametrize("n,s", [(1000, 5000), (50000, 400000)])
def test_chung_lu_gpu_equals_cpu(n, s, gpu_device):
    _same(inputs.chung_lu(n, s, seed=2), inputs.chung_lu(n, s, seed=2, device="cuda"))
