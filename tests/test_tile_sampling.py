"""The row sampler of the full-size GPU parity tests (CPU only)."""

import numpy as np

from gpu_util import tile_rows
from paper_2607_27744_amd import workloads as wl


def test_tile_rows_cover_every_tile():
    # Every request-aligned 128- and 256-row tile and every contiguous
    # 256-row tile of the candidate range holds a sampled row.
    counts = np.array([300, 0, 1, 257, 128, 1000, 5])
    off = wl.offsets_from_counts(counts)
    rows = tile_rows(off, 0)
    for r in range(len(counts)):
        a, b = int(off[r]), int(off[r + 1])
        for t in (128, 256):
            for s in range(a, b, t):
                assert np.any((rows >= s) & (rows < min(s + t, b)))
    n = int(off[-1])
    for s in range(0, n, 256):
        assert np.any((rows >= s) & (rows < min(s + 256, n)))
