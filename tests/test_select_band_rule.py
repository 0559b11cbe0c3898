"""CPU check of the band rule that settles top-k rows the float bound cannot.

The fast selection holds float estimates w^ of the block weights W with
|w^ - W| <= W*dl + eps per block.  For a row whose cut it cannot certify it
marks the blocks whose lower bound exceeds the upper bound of the (m+1)-th
largest w^ as certainly kept, those whose upper bound is below the lower
bound of the m-th largest as certainly dropped, and settles the rest (the
band) by the exact weights.  This test replays that rule on random rows,
near-ties included, and checks that the result is always the exact top m
(App. J's top-k, ties to the lowest block id).
"""
import numpy as np


def band_select(what, W, m, dl, eps):
    """Top-m ids by the band rule; None when the fast bound already settles the row."""
    order = np.argsort(-what, kind="stable")
    a = what[order[m - 1]]
    cnt_ge = int((what >= a).sum())
    below = what[what < a]
    lt = below.max() if len(below) else 0.0
    if cnt_ge == m and a * (1 - dl) - eps > lt * (1 + dl) + eps:
        return None
    wm1 = a if cnt_ge > m else lt
    tin = wm1 * (1 + dl) + eps
    tout = a * (1 - dl) - eps
    sure_in = what * (1 - dl) - eps > tin
    sure_out = what * (1 + dl) + eps < tout
    band = np.nonzero(~sure_in & ~sure_out)[0]
    need = m - int(sure_in.sum())
    assert 0 <= need <= len(band)
    ranked = sorted(band, key=lambda v: (-W[v], v))
    return set(np.nonzero(sure_in)[0]) | set(ranked[:need])


def test_band_rule_gives_the_exact_top_m():
    rng = np.random.default_rng(7)
    checked = 0
    for _ in range(6000):
        CK = int(rng.integers(5, 60))
        m = int(rng.integers(1, CK))
        W = rng.exponential(1.0, CK) ** rng.uniform(1, 4)
        if rng.random() < 0.4:  # near-ties and exact ties
            i, j = rng.integers(0, CK, 2)
            W[i] = W[j] * (1 + rng.uniform(-1e-4, 1e-4) * (rng.random() < 0.7))
        dl = 10 ** rng.uniform(-5, -2)
        eps = 0.0 if rng.random() < 0.5 else 10 ** rng.uniform(-9, -6)
        err = W * rng.uniform(-dl, dl, CK) + rng.uniform(-eps, eps, CK)
        what = (W + err).astype(np.float32).astype(np.float64)
        # the float32 rounding of w^ is part of the estimate's error
        dl_eff = dl + 2.0 ** -23
        sel = band_select(what, W, m, dl_eff, eps)
        if sel is None:
            continue
        checked += 1
        exact = set(sorted(range(CK), key=lambda v: (-W[v], v))[:m])
        assert sel == exact
    assert checked > 100


def test_band_rule_catches_a_planted_mistake():
    # ranking the band by the estimate instead of the exact weight picks the
    # wrong block when the estimate inverts a close pair
    W = np.array([1.0, 0.50001, 0.5, 0.1])
    what = np.array([1.0, 0.5, 0.50001, 0.1])
    dl = 1e-3
    sel = band_select(what, W, 2, dl, 0.0)
    assert sel == {0, 1}
    order_by_estimate = sorted([1, 2], key=lambda v: (-what[v], v))
    assert {0, order_by_estimate[0]} != sel
