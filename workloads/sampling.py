"""Which outputs a full-size parity check compares (no arithmetic of the method).

At full workload sizes the oracle evaluates the convolution one output at a
time, so a check compares a sample of outputs.  The sample is chosen so that
an error confined to one piece of the output is still found:

* ``count`` uniformly random outputs;
* one random output in every (pixel block, col-group) cell, where a pixel
  block is ``block_px`` consecutive output pixels in batch-major order and a
  col-group is N consecutive output channels.  A kernel that computes the
  output in tiles of pixels and col-groups (and, when it splits a tile's
  contraction, adds the parts into that tile) gets at least one sampled
  output in every tile of ``block_px`` pixels or more; when the cells outnumber
  ``cap`` the block is doubled until they do not;
* the corners of the output, the first and last pixel of the first and last
  image in every row of the last (possibly ragged) col-group.
"""
import numpy as np


def sample_outputs(shape, N, count=10000, seed=0, block_px=128, cap=30000):
    """Sorted unique flat NCHW indices into an output of ``shape`` = (B, n, Ho, Wo)."""
    B, n, Ho, Wo = (int(v) for v in shape)
    hw = Ho * Wo
    npix = B * hw
    total = npix * n
    if total == 0:
        return np.zeros(0, np.int64)
    rng = np.random.default_rng(seed)
    parts = [rng.integers(0, total, size=count, dtype=np.int64)]

    G = -(-n // N)
    while -(-npix // block_px) * G > cap and block_px < npix:
        block_px *= 2
    nblk = -(-npix // block_px)
    blk = np.repeat(np.arange(nblk, dtype=np.int64), G)
    grp = np.tile(np.arange(G, dtype=np.int64), nblk)
    lo = blk * block_px
    span = np.minimum(lo + block_px, npix) - lo
    pix = lo + (rng.random(blk.size) * span).astype(np.int64)
    rows = np.minimum(grp * N + N, n) - grp * N
    ch = grp * N + (rng.random(grp.size) * rows).astype(np.int64)
    b, r = np.divmod(pix, hw)
    parts.append((b * n + ch) * hw + r)

    extra = [0, total - 1, (n - 1) * hw, ((B - 1) * n + (n - 1)) * hw + hw - 1]
    for o in range((n - 1) // N * N, n):
        for bb in {0, B - 1}:
            extra += [(bb * n + o) * hw, (bb * n + o) * hw + hw - 1, (bb * n + o) * hw + hw // 2]
    parts.append(np.array(extra, np.int64))
    return np.unique(np.concatenate(parts))
