"""Pins for the oracle's Tier-2 region copy (section 3.4: a captured state is
restored in place before every replay): numpy slice assignment of the same
regions, at odd offsets and lengths, with adjacent and empty regions, in any
order of the region list."""
import numpy as np

import oracle


def _numpy_copy(buf, regions):
    out = buf.copy()
    for d, s, n in regions:
        out[d:d + n] = out[s:s + n].copy()
    return out


def test_copy_regions_equals_numpy_slices():
    rng = np.random.default_rng(31)
    for trial in range(200):
        size = int(rng.integers(64, 20_000))
        buf = rng.integers(0, 256, size=size, dtype=np.uint8)
        half = size // 2
        # destinations in the upper half, sources in the lower half: never overlapping
        cuts = np.sort(rng.choice(np.arange(half, size), size=int(rng.integers(2, 12)), replace=False))
        regions = []
        for lo, hi in zip(cuts[:-1], cuts[1:]):   # adjacent destination ranges
            n = int(hi - lo)
            if trial % 5 == 0 and rng.random() < 0.3:
                n = 0                             # an empty region
            if n <= half:
                regions.append((int(lo), int(rng.integers(0, half - n + 1)), n))
        if trial % 2:
            rng.shuffle(regions)
        want = _numpy_copy(buf, regions)
        got = buf.copy()
        oracle.copy_regions(got, regions)
        assert np.array_equal(got, want), regions
        for d, s, n in regions:                   # and each destination holds its source bytes
            assert np.array_equal(got[d:d + n], buf[s:s + n])


def test_copy_regions_chain_in_order():
    """Regions are applied in list order: a region whose source is an earlier
    region's destination sees the copied bytes."""
    buf = np.arange(64, dtype=np.uint8)
    got = buf.copy()
    oracle.copy_regions(got, [(16, 1, 7), (40, 16, 7)])
    assert np.array_equal(got[16:23], buf[1:8]) and np.array_equal(got[40:47], buf[1:8])
    oracle.copy_regions(got, [])
    assert np.array_equal(got[:16], buf[:16])
