"""Pins of the oracle's closed-form route counts against hand-worked integers."""
import pytest

from golden_io import load
from oracle import cost


@pytest.mark.parametrize("case", load("route_counts.json")["cases"], ids=lambda c: c["name"])
def test_route_counts_match_hand_derivation(case):
    a = (case["d_in"], case["d_out"], case["k_in"], case["k_out"], case["T"])
    assert cost.factored_flops(*a) == case["factored"]
    assert cost.materialized_flops(*a) == case["materialized"]
    if "storage_threshold" in case:
        assert cost.storage_threshold(case["d_in"], case["d_out"]) == pytest.approx(case["storage_threshold"], rel=1e-15)


def test_storage_rule_regimes():
    # factorized smaller iff T < N_i N_o / (N_i + N_o)
    for N_i, N_o in ((8192, 28672), (64, 64), (32, 32)):
        thr = cost.storage_threshold(N_i, N_o)
        for T in (1, int(thr), int(thr) + 1, 4 * int(thr) + 3):
            smaller = cost.storage_factorized(N_i, N_o, T) < cost.storage_materialized(N_i, N_o)
            assert smaller == (T < thr)
    # projected regime: k_a k_g/(k_a+k_g) with k = 64 is 32, far below realistic T
    assert cost.storage_threshold(64, 64) == 32


def test_crossgram_regimes():
    # short sequences / wide layers favour factorized; long sequences favour materialized
    assert cost.crossgram_factorized(8, 1, 32, 4096, 4096) < cost.crossgram_materialized(8, 1, 32, 4096, 4096)
    assert cost.crossgram_factorized(8, 8, 8192, 1024, 1024) > cost.crossgram_materialized(8, 8, 8192, 1024, 1024)
