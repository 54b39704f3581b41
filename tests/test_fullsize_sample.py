"""The full-size parity sample (host logic of tests/test_gpu_fullsize.py):
every 1024-element block of the pass is sampled, the lane positions rotate
through all 1024, and both sides of every 8192-element tile edge are in."""
import numpy as np
import pytest

from test_gpu_fullsize import BLOCK_ELEMS, TILE_ELEMS, _sample


@pytest.mark.parametrize("P", [4096, 1_200_000, 11_700_000, 25_000_000, 124_000_007])
def test_sample_covers_every_block_lane_and_tile_edge(P):
    idx = _sample(P, seed=P)
    assert idx.min() >= 0 and idx.max() < P and np.all(np.diff(idx) > 0)
    nblk = -(-P // BLOCK_ELEMS)
    assert np.array_equal(np.unique(idx // BLOCK_ELEMS), np.arange(nblk))
    if nblk >= BLOCK_ELEMS:
        assert np.unique(idx % BLOCK_ELEMS).size == BLOCK_ELEMS
    edges = np.arange(TILE_ELEMS, P, TILE_ELEMS)
    assert np.all(np.isin(edges, idx)) and np.all(np.isin(edges - 1, idx))
    assert P - 1 in idx
