"""Schedule policies and communication accounting (host only), checked
against values worked out by hand from the policies' definitions."""
import pytest

from paper_2202_06009_amd import schedules as S


def test_kappa_rule_gaps_double_every_kappa_updates():
    assert S.tv_kappa(50, kappa=2) == [0, 1, 2, 4, 6, 10, 14, 22, 30, 46]
    ks = S.tv_kappa(10_000, kappa=16)
    gaps = [b - a for a, b in zip(ks, ks[1:])]
    assert gaps == [2 ** (j // 16) for j in range(len(gaps))]
    assert ks[:17] == list(range(17)) and ks[17] == 18


def test_sync_interval_doubles_after_warmup_and_is_clipped():
    got = S.tu_doubling(40, warmup=4, period=8, H=4)
    assert got == list(range(12)) + [12, 14, 16, 18, 20, 24, 28, 32, 36]
    # H = 16 caps the paper's interval
    got = S.tu_doubling(10_000, warmup=10, period=100, H=16)
    assert max(b - a for a, b in zip(got, got[1:])) == 16


def test_inverse_learning_rate_interval():
    gammas = [1.0] * 4 + [0.5] * 4 + [0.26] * 8 + [0.01] * 40
    got = S.tu_inverse_lr(gammas, H=16)
    # interval 1 at rate 1, 2 at 0.5, 2 at 0.26 (1/0.26 = 3.8), 16 (clipped 64) at 0.01
    assert got == [0, 1, 2, 3, 4, 6, 8, 10, 12, 14, 16, 32, 48]


def test_variance_frozen_once_the_interval_exceeds_one():
    tu = [0, 1, 2, 3, 5, 7, 11]
    assert S.freeze_variance(range(12), tu, 12) == [0, 1, 2, 3]
    assert S.freeze_variance([0, 2, 6], [0, 1, 2, 4, 5, 6], 8) == [0, 2, 6]


def test_communication_counts():
    c = S.communication(10, [0, 1], [0, 1, 2, 4, 8], n_params=1000, chunk=1024)
    assert c["bits_per_param"] == pytest.approx(16 * 2 + 5 * (1 + 32 / 1024))
    assert c["rounds"] == 7 and c["steps_communicating"] == 5
    b = S.one_bit_adam_communication(10, 2, n_params=1000, chunk=1024)
    assert b["bits_per_param"] == pytest.approx(16 * 2 + 8 * (1 + 32 / 1024))
    assert b["rounds"] == 10 and b["steps_communicating"] == 10


def test_paper_policies_communicate_less_than_one_bit_adam():
    """The kind of comparison the paper plots: 0/1 Adam with the kappa rule,
    the doubling interval (H = 16) and the variance freeze against 1-bit Adam
    with a full-precision stage of 15% of the steps."""
    T, warmup, period = 20_000, 1250, 3277
    tu = S.tu_doubling(T, warmup, period)
    tv = S.freeze_variance(S.tv_kappa(T), tu, T)
    ours = S.communication(T, tv, tu, 1, 16384)
    base = S.one_bit_adam_communication(T, int(0.15 * T), 1, 16384)
    assert ours["bits_per_param"] < 0.5 * base["bits_per_param"]
    assert ours["rounds"] < 0.5 * base["rounds"]
    # the interval first exceeds one step a period after the warm-up
    assert all(t < warmup + period for t in tv) and tv[-1] > warmup
