"""Sequence-group shapes of the pipelined decode step (host logic, CPU):
every rule covers the batch exactly once with non-empty groups."""
import pytest

from paper_2509_24626_amd import harness as H


@pytest.mark.parametrize("B", [7, 16, 40, 41, 48, 63, 64, 65, 100, 128, 256, 1000])
def test_ramp_parts_cover_the_batch(B):
    sizes = H.ramp_parts(B)
    assert sum(sizes) == B and min(sizes) >= 1
    if B >= 40:
        assert len(sizes) == 7
        peak = sizes.index(max(sizes))
        # groups grow up to the largest and shrink after it
        assert all(a <= b for a, b in zip(sizes[:peak], sizes[1:peak + 1]))
        assert all(a >= b for a, b in zip(sizes[peak:], sizes[peak + 1:]))


def test_ramp_parts_at_batch_64():
    assert H.ramp_parts(64) == [2, 4, 10, 20, 18, 8, 2]


@pytest.mark.parametrize("B,n", [(1, 1), (5, 3), (16, 4), (64, 6), (64, 8), (48, 5), (3, 7)])
def test_tent_parts_cover_the_batch(B, n):
    sizes = H.tent_parts(B, n)
    assert sum(sizes) == B and min(sizes) >= 1 and len(sizes) == min(n, B)


def test_default_parts():
    assert H.default_parts(64) == H.ramp_parts(64)
    assert H.default_parts(48) == H.ramp_parts(48)
    assert H.default_parts(16) == [2, 3, 5, 6] and H.default_parts(8) == [1, 2, 2, 3]
    for B in range(8, 40):
        sizes = H.default_parts(B)
        assert len(sizes) == 4 and sum(sizes) == B and min(sizes) >= 1
    assert H.default_parts(2) == 1 and H.default_parts(7) == 2 and H.default_parts(1) == 1
