"""The any-size list check used by the full-size parity tests accepts the
oracle's sorted list and rejects each plausible corruption of it (CPU only)."""
import numpy as np
import pytest

from paper_2609_05255_amd import inputs
from parity import check_list_properties, tile_of_ranges


@pytest.fixture(scope="module")
def tiny_lists(orc):
    sc = inputs.make_scene("tiny")
    cam = inputs.make_cameras("tiny")[0]
    pre = orc.preprocess(cam, sc)
    values, tile_of, ranges = orc.bin_sort(cam, pre)
    key = np.where(pre["tiles"] > 0, pre["depth"].astype(np.float32).view(np.uint32), np.uint32(0xFFFFFFFF))
    return dict(values=values, tile_of=tile_of, ranges=ranges, tiles=pre["tiles"], rect=pre["rect"], key=key,
                tiles_x=orc.tile_grid(cam)[0])


def check(d, values=None, tile_of=None):
    check_list_properties(d["values"] if values is None else values, d["tile_of"] if tile_of is None else tile_of,
                          d["tiles"], d["rect"], d["key"], d["tiles_x"])


def test_accepts_oracle_list(tiny_lists):
    d = tiny_lists
    assert d["values"].size > 1000
    check(d)
    assert np.array_equal(tile_of_ranges(d["ranges"], d["values"].size), d["tile_of"])


def test_rejects_swapped_neighbours(tiny_lists):
    d = tiny_lists
    t = d["tile_of"]
    i = int(np.nonzero(t[1:] == t[:-1])[0][0])       # two entries of one tile
    v = d["values"].copy()
    v[i], v[i + 1] = v[i + 1], v[i]
    with pytest.raises(AssertionError):
        check(d, values=v)


def test_rejects_duplicate_and_missing_pair(tiny_lists):
    d = tiny_lists
    t = d["tile_of"]
    i = int(np.nonzero(t[1:] == t[:-1])[0][0])
    v = d["values"].copy()
    v[i + 1] = v[i]                                    # one Gaussian twice, another missing
    with pytest.raises(AssertionError):
        check(d, values=v)


def test_rejects_wrong_tile(tiny_lists):
    d = tiny_lists
    t = d["tile_of"].copy()
    j = int(np.nonzero(t[1:] != t[:-1])[0][0])        # last entry of a tile moved into the next one
    t[j] = t[j + 1]
    with pytest.raises(AssertionError):
        check(d, tile_of=t)


def test_rejects_dropped_pair(tiny_lists):
    d = tiny_lists
    with pytest.raises(AssertionError):
        check(d, values=d["values"][1:], tile_of=d["tile_of"][1:])


def test_rejects_broken_ranges(tiny_lists):
    d = tiny_lists
    r = d["ranges"].copy()
    k = int(np.nonzero(r[:, 1] > r[:, 0])[0][0])
    r[k, 1] -= 1                                       # a gap between two tiles
    with pytest.raises(AssertionError):
        tile_of_ranges(r, d["values"].size)
