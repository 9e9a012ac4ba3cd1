"""The sampled-output selection used by the full-size parity checks (CPU)."""
import numpy as np
import pytest

import workloads


@pytest.mark.parametrize("shape,N", [((64, 256, 56, 56), 32), ((128, 960, 7, 7), 4),
                                     ((3, 72, 9, 7), 32), ((1, 5, 1, 1), 4)])
def test_every_tile_and_col_group_is_sampled(shape, N):
    B, n, Ho, Wo = shape
    idx = workloads.sample_outputs(shape, N, 10000, seed=1)
    total = B * n * Ho * Wo
    assert idx.min() >= 0 and idx.max() < total
    assert np.all(np.diff(idx) > 0)
    assert idx.size >= min(10000, total) * 0.6        # random draws repeat on tiny outputs
    b, rest = np.divmod(idx, n * Ho * Wo)
    o, hw = np.divmod(rest, Ho * Wo)
    pix = b * Ho * Wo + hw
    npix, G = B * Ho * Wo, -(-n // N)
    blk = 128
    while -(-npix // blk) * G > 30000 and blk < npix:
        blk *= 2
    cells = set(zip((pix // blk).tolist(), (o // N).tolist()))
    assert len(cells) == -(-npix // blk) * G
    assert {0, total - 1} <= set(idx.tolist())
    last_group = set(range((n - 1) // N * N, n))
    assert last_group <= set(o.tolist())
