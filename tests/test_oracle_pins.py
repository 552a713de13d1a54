"""The oracle against its pins (CPU only)."""
import pytest

import oracle
import pins


@pytest.mark.parametrize("check", pins.ATTENTION_CHECKS, ids=lambda f: f.__name__)
def test_attention_pin(check):
    check(oracle.attention)


@pytest.mark.parametrize("check", pins.LMHEAD_CHECKS, ids=lambda f: f.__name__)
def test_lmhead_pin(check):
    check(oracle.lmhead)


@pytest.mark.parametrize("check", pins.SELECT_CHECKS, ids=lambda f: f.__name__)
def test_select_pin(check):
    check(oracle.select)


@pytest.mark.parametrize("check", pins.REFRESH_CHECKS, ids=lambda f: f.__name__)
def test_refresh_pin(check):
    check(oracle.refresh)


@pytest.mark.parametrize("check", pins.SCHEDULER_CHECKS, ids=lambda f: f.__name__)
def test_scheduler_pin(check):
    check(oracle.scheduler)
