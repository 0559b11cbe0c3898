"""CPU checks of the parity exemptions: near-ties pass, planted mistakes fail."""
import numpy as np

import parity as PT


def test_topp_mass_tie_exempts_only_the_cut_block():
    # descending weights 0.5, 0.3, 0.1 (+ 0.1 split); p = 0.8 is reached
    # exactly at the second block, so the next block (id 2) may be added
    w = np.array([0.5, 0.3, 0.1, 0.06, 0.04])
    valid = np.ones(5, bool)
    want = {0, 1}
    assert PT.mask_row_exempt(w, valid, "topp", 0.8, {0, 1, 2}, want)
    # dropping a block away from the cut, or adding a far block, is a mistake
    assert not PT.mask_row_exempt(w, valid, "topp", 0.8, {0, 1, 2, 4}, want)
    assert not PT.mask_row_exempt(w, valid, "topp", 0.8, {0, 1, 3}, want)
    assert not PT.mask_row_exempt(w, valid, "topp", 0.8, {0}, want)


def test_topp_previous_prefix_tie_exempts_dropping_the_last_block():
    # cumulative 0.5, 0.8, 0.9: the oracle keeps three blocks for p = 0.8 + 1e-9
    # (0.8 < p), so stopping after two (the last kept block dropped) is a tie
    w = np.array([0.5, 0.3, 0.1, 0.1])
    valid = np.ones(4, bool)
    p = 0.8 + 1e-9
    want = {0, 1, 2}
    assert PT.mask_row_exempt(w, valid, "topp", p, {0, 1}, want)
    assert not PT.mask_row_exempt(w, valid, "topp", p, {0, 2}, want)


def test_value_ties_and_mistakes_topk():
    w = np.array([0.4, 0.2, 0.2 * (1 + 1e-8), 0.1, 0.1])
    valid = np.ones(5, bool)
    want = {0, 2}  # top-2 keeps the larger of the tied pair
    assert PT.mask_row_exempt(w, valid, "topk", 0.4, {0, 1}, want)
    assert not PT.mask_row_exempt(w, valid, "topk", 0.4, {0, 3}, want)
    n_diff, n_bad = PT.compare_masks(w[None, :], np.ones(5, int), np.array([3]), "topk", 0.4,
                                     np.array([2]), np.array([[0, 3, -1, -1, -1]]))
    assert (n_diff, n_bad) == (1, 1)
