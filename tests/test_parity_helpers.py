"""The sampled-parity helpers, checked against what they claim: the
probability that two inverse-CDF draws sharing a uniform differ (Monte
Carlo) and the Poisson quantile (scipy)."""
import numpy as np
import pytest

from tests.parity import draw_split, near_tie_bound


def _index(cdf, u):
    return np.searchsorted(cdf, u, side="right")


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_draw_split_bounds_the_disagreement_of_shared_uniform_draws(seed):
    rng = np.random.default_rng(seed)
    wa = rng.random(50) ** 3
    wb = wa * np.exp(0.05 * rng.normal(size=50))
    ca, cb = np.cumsum(wa) / wa.sum(), np.cumsum(wb) / wb.sum()
    u = rng.random(200_000)
    differ = np.mean(_index(ca, u) != _index(cb, u))
    split = draw_split(wa, wb)
    assert abs(differ - split) <= 4 * np.sqrt(split / len(u)) + 1e-4
    assert 0.0 < split < 0.5
    assert draw_split(wa, wa) == 0.0


def test_draw_split_of_near_one_hot_rows_counts_each_u_once():
    # both rows put almost all mass on token 3; the tails differ everywhere
    wa = np.full(1000, 1e-6); wa[3] = 1.0
    wb = np.full(1000, 2e-6); wb[3] = 1.0
    ca, cb = np.cumsum(wa) / wa.sum(), np.cumsum(wb) / wb.sum()
    u = np.random.default_rng(3).random(400_000)
    differ = np.mean(_index(ca, u) != _index(cb, u))
    assert draw_split(wa, wb) == pytest.approx(differ, abs=2e-3)
    assert draw_split(wa, wb) < 2e-3


def test_draw_split_equals_the_disagreement_for_two_outcomes():
    # two outcomes: the draws differ exactly when u lies between the two CDF values
    assert draw_split([0.3, 0.7], [0.35, 0.65]) == pytest.approx(0.05)


def test_near_tie_bound_is_the_poisson_quantile():
    stats = pytest.importorskip("scipy.stats")
    for mu in (0.0, 0.05, 0.3, 1.0, 2.5, 7.0):
        n = near_tie_bound(mu)
        assert stats.poisson.sf(n, mu) <= 1e-3
        if n > 0:
            assert stats.poisson.sf(n - 1, mu) > 1e-3


def test_bf16_tolerance_scales_only_past_the_papers_depths():
    """The bf16 bound is the stated 2e-2 of the logit range for models of up to
    40 layers (the paper's LLaMA-2 7B / 13B); deeper ones get sqrt(depth / 40)
    of it; fp32 stays absolute."""
    from oracle.model import Tolerance
    t = Tolerance()
    for depth in (0, 4, 32, 40):
        assert t.of("bf16", 10.0, depth) == pytest.approx(0.2)
    assert t.of("bf16", 10.0, 80) == pytest.approx(0.2 * 2 ** 0.5)
    assert t.of("bf16", 10.0, 160) == pytest.approx(0.4)
    assert t.of("f32", 10.0, 80) == 1e-4
