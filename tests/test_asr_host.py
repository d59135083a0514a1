"""Host-side pieces of the reconciliation driver that need no GPU."""
import collections

import pytest

from paper_2605_07325_amd import asr


@pytest.mark.parametrize("per_xcd", [1, 2, 3, 4, 6, 8, 12, 16])
def test_partition_masks_cover_every_xcd_under_both_cu_numberings(per_xcd):
    sec = asr.xcd_spread_cus(per_xcd)
    prim = sorted(set(range(256)) - set(sec))
    assert len(sec) == 8 * per_xcd and len(set(sec)) == len(sec)
    for xcd_of in (lambda c: c // 32, lambda c: c % 8):   # blocked or round-robin numbering
        assert sorted(collections.Counter(map(xcd_of, sec)).values()) == [per_xcd] * 8
        assert sorted(collections.Counter(map(xcd_of, prim)).values()) == [32 - per_xcd] * 8


def test_partition_mask_rejects_sizes_that_cannot_spread():
    for bad in (0, 5, 7, 33):
        with pytest.raises(ValueError):
            asr.xcd_spread_cus(bad)


def test_range_helpers():
    assert asr.rlen([(0, 3), (10, 12)]) == 5
    assert asr.rlen([]) == 0
