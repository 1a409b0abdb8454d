"""The 8-bit slice selection (host logic in the C library): never above the target
fraction, greedy by decreasing size so no unchosen tensor would still fit, and the
end cases."""
import pytest

import paper_2608_11919_amd as lt
import synth


@pytest.mark.parametrize("fraction", [0.0, 0.005, 0.02, 0.1, 0.5, 1.0])
def test_slice_is_greedy_and_bounded(fraction):
    numels = synth.full_3b().numels
    total = sum(numels)
    mask, chosen = lt.lt_select_8bit_slice(numels, fraction)
    assert chosen == sum(n for n, m in zip(numels, mask) if m)
    assert chosen <= fraction * total
    left = fraction * total - chosen
    assert all(n > left for n, m in zip(numels, mask) if not m)  # nothing else fits
    if fraction == 1.0:
        assert all(mask)
    if fraction == 0.0:
        assert not any(mask)


def test_slice_prefers_larger_tensors_then_list_order():
    mask, chosen = lt.lt_select_8bit_slice([10, 30, 30, 5, 25], 0.6)  # target 60 of 100
    assert mask == [False, True, True, False, False] and chosen == 60
    mask, chosen = lt.lt_select_8bit_slice([10, 30, 30, 5, 25], 0.4)  # target 40: first 30, then 10
    assert mask == [True, True, False, False, False] and chosen == 40
