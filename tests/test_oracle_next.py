"""The oracle's threshold update, entropy selection and KV write against their pins."""
import importlib

import pytest

import oracle_pins_next as pins

upd = importlib.import_module("oracle.update")
ent = importlib.import_module("oracle.entropy")
kvc = importlib.import_module("oracle.kv_cache")


@pytest.mark.parametrize("check", pins.UPDATE_CHECKS, ids=lambda c: c.__name__)
def test_update_pins(check):
    check(upd)


@pytest.mark.parametrize("check", pins.ENTROPY_CHECKS, ids=lambda c: c.__name__)
def test_entropy_pins(check):
    check(ent)


@pytest.mark.parametrize("check", pins.KV_CHECKS, ids=lambda c: c.__name__)
def test_kv_pins(check):
    check(kvc)
