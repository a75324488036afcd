"""Pins of the attention oracle (CPU only)."""
import pytest

import oracle
import oracle_pins as pins


def test_brute_force_agrees():
    pins.check_brute_force(oracle, oracle.brute_window_attention)


@pytest.mark.parametrize("check", pins.ATTENTION_CHECKS, ids=lambda c: c.__name__)
def test_attention_pin(check):
    check(oracle)


def test_empty_window_rows():
    case = pins.small_case(41, batch=2, prefix=(8, 0), window_lens=[0, 16])
    o = oracle.window_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                                case.prefix_lens, case.window_lens, case.block_size)
    assert o.shape == (16, case.num_q_heads, case.head_dim)
