"""Pins of the attention oracle (CPU only)."""
import numpy as np
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


@pytest.mark.parametrize("seed", range(12))
def test_brute_force_random_small_shapes(seed):
    """Seeded random small shapes (prefix 0..40, 1..3 blocks of 2..8, 1..2 KV
    heads, 1..3 query heads each, D 4 or 8, ragged windows including empty
    ones): the oracle equals the scalar-loop brute force in both mask modes."""
    rng = np.random.default_rng(1000 + seed)
    batch = int(rng.integers(1, 4))
    B = int(rng.choice([2, 4, 8]))
    k = int(rng.integers(1, 4))
    Hkv = int(rng.integers(1, 3))
    Hq = Hkv * int(rng.integers(1, 4))
    D = int(rng.choice([4, 8]))
    prefix = [int(x) for x in rng.integers(0, 41, size=batch)]
    windows = [int(x) * B for x in rng.integers(0, k + 1, size=batch)]
    windows[int(rng.integers(batch))] = k * B          # at least one window row
    case = pins.small_case(2000 + seed, batch=batch, B=B, k=k, Hq=Hq, Hkv=Hkv, D=D, prefix=prefix,
                           window_lens=windows)
    for mode, bidir in ((oracle.MASK_BIDIR, True), (oracle.MASK_BLOCK_CAUSAL, False)):
        o = oracle.window_attention(case.q, case.k_pages, case.v_pages, case.page_table,
                                    case.prefix_lens, case.window_lens, B, mode)
        r = oracle.brute_window_attention(case.q, case.k_pages, case.v_pages, case.page_table, case.prefix_lens,
                                   case.window_lens, B, bidirectional=bidir)
        pins.assert_close(o, r, 1e-12, f"seed {seed} bidir={bidir} P={prefix} W={windows}")
