"""The asynchronous quality gate's re-run rule (tests/gpu_common.py), on made-up log-likelihoods."""
import pytest

from gpu_common import gated, ll_gate


def runs(values):
    it = iter(values)
    calls = []

    def run():
        calls.append(1)
        return next(it)

    return run, calls


def test_gain_fraction_is_the_share_of_the_oracle_gain():
    assert ll_gate(-10.05, -10.0, -10.5) == pytest.approx(0.9)


def test_a_first_run_inside_the_gate_is_the_only_one():
    run, calls = runs([-10.02, -11.0])
    assert gated(run, -10.0, -10.5, 0.9) == pytest.approx(0.96)
    assert len(calls) == 1


def test_one_miss_is_run_again():
    run, calls = runs([-10.2, -10.03])
    assert gated(run, -10.0, -10.5, 0.9) == pytest.approx(0.94)
    assert len(calls) == 2


@pytest.mark.parametrize("values", [[-10.2, -10.2], [-10.2, -10.2001], [-9.0, -9.0]])
def test_two_misses_fail(values):
    run, calls = runs(values)
    with pytest.raises(AssertionError):
        gated(run, -10.0, -10.5, 0.9)
    assert len(calls) == 2
